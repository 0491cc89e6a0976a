"""The C ABI boundary on the host: the library loads, exports what include/forge.h declares,
and every documented validation error is returned before any HIP call.

Pointers here are fake addresses: validation never dereferences them.  No test makes a
call whose arguments are all valid (that would launch a kernel on a GPU machine).
"""
import ctypes
import json
import os

import pytest

from paper_2606_22932_amd import accounting, forge

OK, NULLP, SHAPE, UNSUP, HYPER, DTYPE, MISAL, ALIAS, NODEV, LAUNCH = range(10)
F32, BF16, I8 = 0, 1, 2
HP = dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, wd=0.1, step=1)

GiB = 1 << 30
# well separated, 256-byte aligned fake device addresses
BASE = {k: (i + 1) * 8 * GiB for i, k in enumerate(["X", "dY", "W", "m", "v", "ms", "vs", "G"])}


def lib():
    return forge.lib()


def call_step(T=64, d_in=128, d_out=256, md=BF16, **over):
    a = dict(BASE)
    a.update({k: v for k, v in over.items() if k in a})
    hp = dict(HP)
    hp.update({k: v for k, v in over.items() if k in hp})
    return lib().forge_linear_step(a["X"], a["dY"], a["W"], a["m"], a["v"], a["ms"], a["vs"], T, d_in, d_out,
                                   md, hp["lr"], hp["beta1"], hp["beta2"], hp["eps"], hp["wd"], hp["step"], None)


def call_unfused(T=64, d_in=128, d_out=256, md=BF16, gd=0, **over):
    a = dict(BASE)
    a.update({k: v for k, v in over.items() if k in a})
    hp = dict(HP)
    hp.update({k: v for k, v in over.items() if k in hp})
    return lib().forge_linear_step_unfused(a["X"], a["dY"], a["W"], a["m"], a["v"], a["ms"], a["vs"], T, d_in,
                                           d_out, md, hp["lr"], hp["beta1"], hp["beta2"], hp["eps"], hp["wd"],
                                           hp["step"], a["G"], gd, None)


def test_library_exports_every_header_function():
    names = forge.header_functions()
    assert set(names) >= {"forge_linear_step", "forge_linear_step_unfused", "forge_wgrad", "forge_adamw",
                          "forge_status_string", "forge_query_tile"}
    L = lib()
    for n in names:
        assert hasattr(L, n), n


def test_status_strings():
    for code in range(12):
        s = forge.forge_status_string(code)
        assert s.startswith(forge.STATUS[code])
    assert "unknown" in forge.forge_status_string(99)


def test_query_tile():
    assert forge.forge_query_tile(512, 4096, 4096, BF16) == (128, 128, 32)
    assert forge.forge_query_tile(4096, 4096, 4096, BF16) == (128, 128, 32)   # one tile at every T
    rows, cols, tk = forge.forge_query_tile(512, 4096, 14336, I8)
    assert rows == 256            # an int8 tile is exactly one scale block tall
    assert forge.forge_query_tile(512, 4096, 4096, 3)[1] % 64 == 0   # row-block int8: whole 64-wide blocks
    r = ctypes.c_int32()
    assert lib().forge_query_tile(512, 64, 64, 7, ctypes.byref(r), None, None) == DTYPE
    assert lib().forge_query_tile(-1, 64, 64, BF16, ctypes.byref(r), None, None) == SHAPE
    assert lib().forge_query_tile(512, 64, -8, BF16, None, None, None) == SHAPE


def test_dtype_errors():
    assert call_step(md=5) == DTYPE
    assert call_step(md=-1) == DTYPE
    assert call_unfused(gd=2) == DTYPE
    assert lib().forge_wgrad(BASE["X"], BASE["dY"], BASE["G"], 8, 8, 8, 5, None) == DTYPE


def test_shape_errors():
    assert call_step(T=-1) == SHAPE
    assert call_step(d_in=-8) == SHAPE
    assert call_step(d_out=-8) == SHAPE
    assert call_step(d_in=12) == UNSUP
    assert call_step(d_out=260) == UNSUP
    assert call_step(d_in=1 << 16, d_out=1 << 16) == UNSUP          # 2^32 elements


def test_empty_matrix_is_a_noop():
    assert call_step(d_in=0, X=0, dY=0, W=0, m=0, v=0) == OK
    assert call_step(d_out=0, X=0, dY=0, W=0, m=0, v=0) == OK
    assert lib().forge_wgrad(0, 0, 0, 5, 0, 8, 0, None) == OK


def test_null_pointer_errors():
    assert call_step(W=0) == NULLP
    assert call_step(m=0) == NULLP
    assert call_step(v=0) == NULLP
    assert call_step(X=0) == NULLP
    assert call_step(dY=0) == NULLP
    assert call_step(md=I8, ms=0) == NULLP
    assert call_step(md=I8, vs=0) == NULLP
    assert call_unfused(G=0) == NULLP
    assert lib().forge_wgrad(BASE["X"], BASE["dY"], 0, 8, 8, 8, 0, None) == NULLP
    assert lib().forge_adamw(0, 0, BASE["W"], BASE["m"], BASE["v"], 0, 0, 8, 8, BF16, 1e-3, 0.9, 0.999,
                             1e-8, 0.1, 1, None) == NULLP


def test_hyperparameter_errors():
    assert call_step(step=0) == HYPER
    assert call_step(step=-3) == HYPER
    assert call_step(beta1=1.0) == HYPER
    assert call_step(beta2=-0.1) == HYPER
    assert call_step(eps=0.0) == HYPER
    assert call_step(lr=-1e-3) == HYPER
    assert call_step(lr=float("nan")) == HYPER
    assert call_step(wd=float("inf")) == HYPER


def test_alignment_errors():
    assert call_step(W=BASE["W"] + 2) == MISAL
    assert call_step(X=BASE["X"] + 8) == MISAL
    assert call_step(md=I8, ms=BASE["ms"] + 4) == MISAL
    assert call_unfused(G=BASE["G"] + 2) == MISAL


def test_aliasing_errors():
    P = 128 * 256
    assert call_step(m=BASE["W"] + 16) == ALIAS                  # m overlaps W
    assert call_step(v=BASE["m"] + 2 * P - 16) == ALIAS          # v starts inside m (bf16 m)
    assert call_step(W=BASE["X"]) == ALIAS                       # output overlaps an input
    assert call_step(W=BASE["dY"] + 16) == ALIAS
    assert call_step(md=I8, vs=BASE["ms"]) == ALIAS
    assert call_unfused(G=BASE["W"]) == ALIAS
    assert call_unfused(G=BASE["X"]) == ALIAS
    # adjacent, non-overlapping buffers are fine up to the device check
    if not _gpu_visible():
        assert call_step(m=BASE["W"] + 2 * P) == NODEV


def _gpu_visible():
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:
        return False


@pytest.mark.skipif(_gpu_visible(), reason="on a GPU machine a valid call would launch on fake pointers")
def test_valid_arguments_reach_the_device_check():
    assert call_step() == NODEV
    assert call_step(T=0, X=0, dY=0) == NODEV


def test_paper_bytes_per_parameter():
    """Sec. 2.2: a standard bf16 step streams 16 B/param (gradient, both moments and the
    weight, each written once and read once); the fused step moves 12."""
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "bytes_per_param.json")))
    T, d = 0, 4096
    P = d * d
    assert accounting.fused_bytes(T, d, d, "bf16") / P == g["fused_bf16"]
    assert accounting.unfused_bytes(T, d, d, "bf16", "bf16") / P == g["standard_bf16"]
    assert g["standard_bf16"] / g["fused_bf16"] == pytest.approx(g["memory_bound_speedup_bound"], abs=0.005)  # printed to 2 decimals


def test_encoding_bytes_per_parameter():
    """The state each encoding moves per parameter, read once and written once: W (bf16 2 B,
    fp8 1 B) and the two moments (bf16 2 B, 8-bit 1 B), plus X and dY once per matrix and
    the int8 scales; fp8 rings are per tensor and not counted."""
    T, d_out, d_in = 512, 4096, 14336
    P = d_out * d_in
    xy = 2 * T * (d_in + d_out)
    assert accounting.fused_bytes(T, d_in, d_out, "fp8") == 8 * P + xy
    assert accounting.fused_bytes(T, d_in, d_out, "bf16", "fp8") == 10 * P + xy
    assert accounting.fused_bytes(T, d_in, d_out, "fp8", "fp8") == 6 * P + xy
    assert accounting.fused_bytes(T, d_in, d_out, "i8") == 8 * P + xy + 16 * (d_out // 256) * d_in
    assert accounting.fused_bytes(T, d_in, d_out, "i8r64") == 8 * P + xy + 16 * d_out * (d_in // 64)


def test_random_fp8_state_is_finite_e4m3_with_rings():
    import torch
    from paper_2606_22932_amd import synth
    wl = synth.WORKLOADS["mlp_wfp8_fp8"]
    mat = synth.Matrix("t", 96, 160, 3)
    W, w_ring, m, m_ring, v, v_ring = synth.random_fp8_state(mat, wl)
    for t in (W, m, v):
        assert t.dtype == torch.float8_e4m3fn and tuple(t.shape) == (96, 160)
        assert torch.isfinite(t.float()).all()            # no 0x7F / 0xFF (NaN) codes
    assert (v.view(torch.uint8) < 0x80).all()              # sqrt(v) codes are non-negative
    assert (m.view(torch.uint8) >= 0x80).any() and (W.view(torch.uint8) >= 0x80).any()
    for r, a in ((w_ring, 3 * wl.w_std), (m_ring, 3 * wl.m_std), (v_ring, 3 * wl.v_std ** 0.5)):
        assert r.dtype == torch.float32 and r.numel() == 4 and torch.allclose(r, torch.full((4,), a))
    none = synth.random_fp8_state(mat, synth.WORKLOADS["mlp"])
    assert all(t is None for t in none)


# ----------------------------------------------------------------------------- grouped step

def _mat(i, d_in=128, d_out=256, **over):
    """Fake descriptor of matrix i: its own X, dY, W, m, v, scales, 1 GiB apart."""
    base = (100 + 16 * i) * GiB
    f = dict(X=base, dY=base + GiB, W=base + 2 * GiB, m=base + 3 * GiB, v=base + 4 * GiB,
             ms=base + 5 * GiB, vs=base + 6 * GiB, d_in=d_in, d_out=d_out)
    f.update(over)
    return forge.forge_matrix(f["X"], f["dY"], f["W"], f["m"], f["v"], f["ms"], f["vs"], f["d_in"], f["d_out"])


def call_group(mats, T=64, md=BF16, n=None, **over):
    hp = dict(HP)
    hp.update(over)
    arr = (forge.forge_matrix * max(1, len(mats)))(*mats)
    return lib().forge_linear_step_grouped(arr, len(mats) if n is None else n, T, md, hp["lr"], hp["beta1"],
                                           hp["beta2"], hp["eps"], hp["wd"], hp["step"], None)


def test_group_count_and_null_errors():
    assert lib().forge_linear_step_grouped(None, 1, 64, BF16, 1e-3, 0.9, 0.999, 1e-8, 0.1, 1, None) == NULLP
    assert call_group([_mat(0)], n=0) == SHAPE
    assert call_group([_mat(i) for i in range(forge.FORGE_MAX_GROUP + 1)]) == SHAPE
    assert call_group([_mat(0)], md=9) == DTYPE


def test_group_checks_every_matrix():
    assert call_group([_mat(0), _mat(1, d_in=12)]) == UNSUP
    assert call_group([_mat(0), _mat(1, W=0)]) == NULLP
    assert call_group([_mat(0), _mat(1, m=(116 * GiB) + 3 * GiB + 2)]) == MISAL
    assert call_group([_mat(0), _mat(1, v=(116 * GiB) + 2 * GiB + 16)]) == ALIAS   # v inside W, same matrix
    assert call_group([_mat(0), _mat(1)], step=0) == HYPER


def test_group_aliasing_across_matrices():
    m0 = _mat(0)
    # the state of matrix 1 overlapping the state of matrix 0
    assert call_group([m0, _mat(1, W=m0.m + 64)]) == ALIAS
    # the state of matrix 1 overlapping the input of matrix 0
    assert call_group([m0, _mat(1, v=m0.X)]) == ALIAS
    assert call_group([m0, _mat(1, W=m0.dY + 16)]) == ALIAS


def test_group_all_empty_is_a_noop():
    assert call_group([_mat(0, d_in=0), _mat(1, d_out=0)]) == OK


@pytest.mark.skipif(_gpu_visible(), reason="on a GPU machine a valid call would launch on fake pointers")
def test_group_valid_arguments_reach_the_device_check():
    # q, k, v style: three matrices sharing X (read-only inputs may be shared)
    m0 = _mat(0)
    assert call_group([m0, _mat(1, X=m0.X), _mat(2, X=m0.X)]) == NODEV
    assert call_group([_mat(0), _mat(1, d_in=0)], T=0) == NODEV


# ----------------------------------------------------------------------------- input gradient and backward

DX = 60 * GiB   # fake dX, apart from every other fake tensor


def call_input_grad(T=64, d_in=128, d_out=256, dY=BASE["dY"], W=BASE["W"], dX=DX):
    return lib().forge_input_grad(dY, W, dX, T, d_in, d_out, None)


def call_backward(T=64, d_in=128, d_out=256, md=BF16, dX=DX, **over):
    a = dict(BASE)
    a.update({k: v for k, v in over.items() if k in a})
    hp = dict(HP)
    hp.update({k: v for k, v in over.items() if k in hp})
    return lib().forge_linear_backward(a["X"], a["dY"], a["W"], a["m"], a["v"], a["ms"], a["vs"], dX, T, d_in,
                                       d_out, md, hp["lr"], hp["beta1"], hp["beta2"], hp["eps"], hp["wd"],
                                       hp["step"], None)


def call_backward_group(mats, T=64, md=BF16, n=None, dX=DX, **over):
    hp = dict(HP)
    hp.update(over)
    arr = (forge.forge_matrix * max(1, len(mats)))(*mats)
    return lib().forge_linear_backward_grouped(arr, len(mats) if n is None else n, T, dX, md, hp["lr"],
                                               hp["beta1"], hp["beta2"], hp["eps"], hp["wd"], hp["step"], None)


def test_input_grad_errors():
    assert call_input_grad(T=-1) == SHAPE
    assert call_input_grad(d_in=12) == UNSUP
    assert call_input_grad(d_out=(1 << 31) // 64 + 8) == UNSUP           # dY past 2^31 elements
    assert call_input_grad(dX=0) == NULLP
    assert call_input_grad(dY=0) == NULLP
    assert call_input_grad(W=0) == NULLP
    assert call_input_grad(dX=DX + 8) == MISAL
    assert call_input_grad(W=BASE["W"] + 2) == MISAL
    assert call_input_grad(dX=BASE["dY"] + 64) == ALIAS
    assert call_input_grad(dX=BASE["W"] - 16) == ALIAS                   # dX's tail runs into W


def test_input_grad_empty_is_a_noop():
    # nothing to write: no pointer is read
    assert call_input_grad(T=0, dY=0, W=0, dX=0) == OK
    assert call_input_grad(d_in=0, dY=0, W=0, dX=0) == OK


@pytest.mark.skipif(_gpu_visible(), reason="on a GPU machine a valid call would launch on fake pointers")
def test_input_grad_valid_arguments_reach_the_device_check():
    assert call_input_grad() == NODEV
    assert call_input_grad(d_out=0, dY=0, W=0) == NODEV                  # zero fill of dX


def test_backward_errors():
    assert call_backward(md=7) == DTYPE
    assert call_backward(d_out=12) == UNSUP
    assert call_backward(W=0) == NULLP
    assert call_backward(step=0) == HYPER
    assert call_backward(dX=0) == NULLP
    assert call_backward(dX=DX + 4) == MISAL
    for name in ("X", "dY", "W", "m", "v"):
        assert call_backward(dX=BASE[name] + 32) == ALIAS, name
    assert call_backward(md=I8, dX=BASE["vs"]) == ALIAS
    # the step's own aliasing rules still apply
    assert call_backward(m=BASE["X"]) == ALIAS


def test_backward_empty_cases():
    assert call_backward(T=0, d_in=0, dX=0) == OK
    # T == 0: dX is empty (may be NULL); the zero-gradient step still validates its state
    assert call_backward(T=0, dX=0, W=0) == NULLP


def test_backward_group_errors():
    assert lib().forge_linear_backward_grouped(None, 1, 64, DX, BF16, 1e-3, 0.9, 0.999, 1e-8, 0.1, 1, None) == NULLP
    assert call_backward_group([_mat(0)], n=0) == SHAPE
    assert call_backward_group([_mat(0), _mat(1, d_in=256)]) == SHAPE      # members disagree on d_in
    assert call_backward_group([_mat(0), _mat(1, d_in=0, d_out=0)]) == SHAPE
    m0 = _mat(0)
    assert call_backward_group([m0, _mat(1, X=m0.X)], dX=0) == NULLP
    assert call_backward_group([m0, _mat(1, X=m0.X)], dX=m0.X) == ALIAS
    m1 = _mat(1, X=m0.X)
    assert call_backward_group([m0, m1], dX=m1.dY + 16) == ALIAS
    assert call_backward_group([m0, m1], md=I8, dX=m1.v_scale) == ALIAS


@pytest.mark.skipif(_gpu_visible(), reason="on a GPU machine a valid call would launch on fake pointers")
def test_backward_valid_arguments_reach_the_device_check():
    assert call_backward() == NODEV
    assert call_backward(d_out=0) == NODEV                               # dX zero-filled, no step
    m0 = _mat(0)
    assert call_backward_group([m0, _mat(1, X=m0.X, d_out=64), _mat(2, X=m0.X, d_out=0)]) == NODEV
    assert call_backward_group([_mat(0, d_out=0)]) == NODEV


# ----------------------------------------------------------------------------- update rules

INVOPT = 10
OPT = forge.OPTIMIZERS


def call_opt(opt="sgd_momentum", T=64, d_in=128, d_out=256, md=BF16, hp=None, step=1, **over):
    a = dict(BASE)
    a.update({k: v for k, v in over.items() if k in a})
    h = forge.forge_hparams(1e-3, 0.9, 0.99, 1e-8, 0.01, 0.0, 0.004)
    for k, v in (hp or {}).items():
        setattr(h, k, v)
    code = OPT[opt] if isinstance(opt, str) else opt
    return lib().forge_linear_step_opt(a["X"], a["dY"], a["W"], a["m"], a["v"], T, d_in, d_out, code, md,
                                       None if over.get("null_hp") else ctypes.byref(h), step, None)


def test_opt_code_dtype_and_hp_errors():
    assert call_opt(opt=99) == INVOPT
    assert call_opt(opt=-1) == INVOPT
    assert call_opt(md=I8) == DTYPE
    assert call_opt(md=5) == DTYPE
    assert call_opt(null_hp=True) == NULLP
    assert call_opt(d_in=12) == UNSUP


def test_opt_state_pointers_follow_the_rule():
    assert call_opt("sgd_momentum", m=0) == NULLP
    assert call_opt("nadam", v=0) == NULLP
    assert call_opt("adamw", W=0) == NULLP
    assert call_opt("sgd_momentum", m=BASE["m"] + 4) == MISAL
    assert call_opt("lion", m=BASE["W"] + 64) == ALIAS
    assert call_opt("radam", v=BASE["m"] + 16) == ALIAS
    assert call_opt("adagrad", m=BASE["dY"]) == ALIAS
    assert call_opt("muon_accumulate", m=BASE["X"] + 32) == ALIAS


def test_opt_hyperparameters_checked_per_rule():
    assert call_opt(step=0) == HYPER
    assert call_opt(hp=dict(lr=-1.0)) == HYPER
    assert call_opt(hp=dict(weight_decay=float("nan"))) == HYPER
    assert call_opt("sgd_momentum", hp=dict(beta1=1.0)) == HYPER
    assert call_opt("nadam", hp=dict(beta2=1.0)) == HYPER
    assert call_opt("nadam", hp=dict(momentum_decay=-1.0)) == HYPER
    assert call_opt("adagrad", hp=dict(lr_decay=-0.1)) == HYPER
    assert call_opt("adagrad", hp=dict(eps=0.0)) == HYPER
    assert call_opt("rmsprop", hp=dict(beta2=-0.5)) == HYPER
    assert call_opt("lion", hp=dict(beta1=1.5)) == HYPER
    assert call_opt("muon_accumulate", hp=dict(beta1=1.5)) == HYPER


def test_opt_empty_is_a_noop():
    assert call_opt(d_in=0) == OK
    assert call_opt("sgd", d_out=0, W=0) == OK


@pytest.mark.skipif(_gpu_visible(), reason="on a GPU machine a valid call would launch on fake pointers")
def test_opt_valid_arguments_reach_the_device_check():
    for name in OPT:
        assert call_opt(name) == NODEV, name
    # rules read only the fields and tensors they use
    assert call_opt("sgd", m=0, v=0, hp=dict(beta1=5.0, eps=0.0)) == NODEV
    assert call_opt("muon_accumulate", W=0, v=0, hp=dict(beta1=1.0)) == NODEV
    assert call_opt("sgd_momentum", v=0, hp=dict(beta2=7.0)) == NODEV


# ----------------------------------------------------------------------------- int8, 64-wide row blocks

I8R64 = 3


def test_i8_row64_dtype_and_scale_pointers():
    assert call_step(md=I8R64, ms=0) == NULLP
    assert call_step(md=I8R64, vs=BASE["vs"] + 4) == MISAL
    assert call_step(md=5) == DTYPE
    # the rule API takes fp32 / bf16 state only
    assert call_opt("adamw", md=I8R64) == DTYPE


@pytest.mark.skipif(_gpu_visible(), reason="on a GPU machine a valid call would launch on fake pointers")
def test_i8_row64_scale_extent_is_the_row_layout():
    """d_in 128, d_out 256: row-block scales are 256 x 2 fp32 (2 KiB), column-block ones
    1 x 128 (512 B).  v_scale 1 KiB after m_scale overlaps only in the row layout."""
    vs = BASE["ms"] + 1024
    assert call_step(md=I8R64, vs=vs) == ALIAS
    assert call_step(md=I8, vs=vs) == NODEV
    assert call_step(md=I8R64) == NODEV
    assert call_unfused(md=I8R64) == NODEV


# ----------------------------------------------------------------------------- fp8 encodings

FP8 = 4


def call_wfp8(T=64, d_in=128, d_out=256, md=BF16, w_amax=60 * GiB + 1024, **over):
    a = dict(BASE)
    a.update({k: v for k, v in over.items() if k in a})
    hp = dict(HP)
    hp.update({k: v for k, v in over.items() if k in hp})
    return lib().forge_linear_step_wfp8(a["X"], a["dY"], a["W"], w_amax, a["m"], a["v"], a["ms"], a["vs"], T, d_in,
                                        d_out, md, hp["lr"], hp["beta1"], hp["beta2"], hp["eps"], hp["wd"],
                                        hp["step"], None)


def test_fp8_moment_rings_are_checked():
    assert call_step(md=FP8, ms=0) == NULLP
    assert call_step(md=FP8, vs=BASE["vs"] + 8) == MISAL
    assert call_step(md=FP8, vs=BASE["ms"]) == ALIAS               # the two 16-byte rings overlap
    assert call_adamw_dtype(FP8) == DTYPE
    assert call_unfused(md=FP8) == DTYPE


def call_adamw_dtype(md):
    a = BASE
    return lib().forge_adamw(a["G"], 0, a["W"], a["m"], a["v"], a["ms"], a["vs"], 128, 256, md, 1e-3, 0.9, 0.999,
                             1e-8, 0.1, 1, None)


def test_fp8_weight_entry_point_errors():
    assert call_wfp8(md=0) == DTYPE
    assert call_wfp8(md=I8) == DTYPE
    assert call_wfp8(w_amax=0) == NULLP
    assert call_wfp8(w_amax=60 * GiB + 4) == MISAL
    assert call_wfp8(md=FP8, ms=0) == NULLP
    assert call_wfp8(w_amax=BASE["W"] + 64) == ALIAS
    assert call_wfp8(m=BASE["W"] + 128 * 256 - 16) == ALIAS       # fp8 W is 1 byte per element
    assert call_wfp8(step=0) == HYPER
    assert call_wfp8(d_in=0) == OK


@pytest.mark.skipif(_gpu_visible(), reason="on a GPU machine a valid call would launch on fake pointers")
def test_fp8_valid_arguments_reach_the_device_check():
    assert call_step(md=FP8) == NODEV
    assert call_wfp8() == NODEV
    assert call_wfp8(md=FP8) == NODEV
    assert call_wfp8(m=BASE["W"] + 128 * 256) == NODEV           # right after a 1-byte-per-element W


def call_noalloc(T=64, d_in=128, d_out=256, md=BF16, gd=0, **over):
    a = dict(BASE)
    a.update({k: v for k, v in over.items() if k in a})
    hp = dict(HP)
    hp.update({k: v for k, v in over.items() if k in hp})
    return lib().forge_linear_step_unfused_noalloc(a["X"], a["dY"], a["W"], a["m"], a["v"], a["ms"], a["vs"], T,
                                                   d_in, d_out, md, hp["lr"], hp["beta1"], hp["beta2"], hp["eps"],
                                                   hp["wd"], hp["step"], gd, None)


def test_noalloc_refuses_gradients_beyond_the_buffer():
    """The fixed buffer holds FORGE_SCRATCH_BYTES: d_in * d_out * (2 or 4 bytes) beyond it is
    FORGE_ERR_SCRATCH_LIMIT, refused on the host before any other pointer or device check."""
    SCRATCH = 11
    assert forge.FORGE_SCRATCH_BYTES == 64 << 20
    assert call_noalloc(d_in=8192, d_out=4104, gd=0) == SCRATCH           # 67,239,936 B of bf16
    assert call_noalloc(d_in=4096, d_out=4104, gd=1) == SCRATCH           # fp32
    assert call_noalloc(d_in=4096, d_out=4104, gd=1, W=0) == SCRATCH      # before the pointer checks
    # exactly the buffer passes the size check (the invalid step is caught after it, so no
    # call here gets as far as a launch)
    assert call_noalloc(d_in=8192, d_out=4096, gd=0, step=0) == HYPER
    assert call_noalloc(d_in=4096, d_out=4096, gd=1, step=0) == HYPER
    # the other rules are those of forge_linear_step_unfused
    assert call_noalloc(gd=2) == DTYPE
    assert call_noalloc(md=4) == DTYPE
    assert call_noalloc(W=0) == NULLP
    assert call_noalloc(step=0) == HYPER
    assert call_noalloc(W=BASE["W"] + 2) == MISAL
    assert call_noalloc(W=BASE["X"]) == ALIAS
    assert call_noalloc(d_out=0) == OK


def test_library_has_no_undefined_internal_symbols():
    """Every kernel launch stub the library references is defined in it (a hipcc build that
    drops a template kernel's host stub would fail to load only when that path is used)."""
    import shutil
    import subprocess
    from paper_2606_22932_amd import build
    nm = shutil.which("nm")
    if nm is None:
        pytest.skip("nm not available")
    out = subprocess.run([nm, "-D", "--undefined-only", build.LIB], capture_output=True, text=True, check=True).stdout
    assert "forge_impl" not in out, out


def test_missing_library_fails_loudly():
    """Without the built HIP library every entry point raises: there is no CPU or PyTorch
    fallback.  Run in a child process so that this process keeps its loaded library."""
    import subprocess
    import sys
    code = (
        "import torch\n"
        "from paper_2606_22932_amd import build, forge\n"
        "build.LIB = '/nonexistent/libforge.so'\n"
        "for f in (forge.lib, lambda: forge.forge_status_string(0),\n"
        "          lambda: forge.forge_query_tile(512, 4096, 4096, 1)):\n"
        "    try:\n"
        "        f()\n"
        "    except RuntimeError as e:\n"
        "        assert 'not built' in str(e) and 'no non-HIP fallback' in str(e), e\n"
        "    else:\n"
        "        raise SystemExit('an entry point ran without the library')\n"
        "x, w = torch.zeros(4, 8, dtype=torch.bfloat16), torch.zeros(8, 8, dtype=torch.bfloat16)\n"
        "try:\n"
        "    forge.forge_linear_step(x, x, w, w.clone(), w.clone(), lr=1e-3, beta1=0.9, beta2=0.999,\n"
        "                            eps=1e-8, weight_decay=0.0, step=1)\n"
        "except Exception as e:\n"
        "    print('step raised', type(e).__name__)\n"
        "else:\n"
        "    raise SystemExit('the step ran on host tensors without the library')\n"
        "print('raised')\n")
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    res = subprocess.run([sys.executable, "-c", code], cwd=root, capture_output=True, text=True, timeout=300)
    assert res.returncode == 0 and "raised" in res.stdout, res.stdout + res.stderr
