"""GPU parity of the fp8 encodings: fp8 moments (m and sqrt(v) as E4M3 with per-tensor delayed
scales), fp8 weights, and both, against the oracle.

Shapes: ragged and multi-tile ones, the smallest legal shape, and the full Llama-3.1-8B
o_proj shape (T=512, 4096 x 4096), where the per-tensor amax is a maximum over the records
of 4096 waves, and the MLP down projection (4096 x 14336, 14336 waves), the shape bench.py
times the fp8 encodings on.  Three consecutive steps from a cold start exercise the whole amax ring
(decode with slot (t-2)%4, encode with (t-1)%4, record into t%4, clear (t+1)%4).  Each step
the oracle starts from the GPU's own state (teacher forcing), so that a rounding tie decided
differently in one step does not compound.

The bar: bf16 tensors as everywhere else (bf16 m and v with the windows of the kernel's
fp32 error, G's included); amax slots within 1e-5 relative (the kernel's
fp32 values against the oracle's fp64 values rounded to fp32); cleared slots exactly zero;
E4M3 codes equal, except
* the adjacent code where the oracle's fp32 quotient x/s lies within 1e-3 (relative) of the
  midpoint between the two values (a tie the kernel's fp32 value may round the other way);
* a code within the range the oracle itself produces when G moves by its fp32 accumulation
  bound E = T 2^-24 |dY|^T |X| (the oracle run at G - E and G + E).  The kernel's G is an
  fp32 sum in some order; where |G| is close to that error, near G = 0, the step's
  g / (|g| + eps) shape lets it move the weight by up to lr.  Over the 16.7M elements of
  the full shape a few such elements occur.
"""
import numpy as np
import pytest
import torch

import oracle
from compare import check_moment, check_weight, moment_windows
from gpu_util import bits, gemm_error_bound
from paper_2606_22932_amd import forge, synth

pytestmark = pytest.mark.gpu

HP = dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.1)


def _say(*a):
    print(*a, flush=True)


def codes(t):
    return t.detach().cpu().contiguous().view(torch.uint8).numpy().copy()


def fp8_tensor(a, device="cuda"):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.uint8)).view(torch.float8_e4m3fn).to(device)


def check_e4m3(gpu, ora, quot, name, rel=1e-3, quot_alts=()):
    """E4M3 codes: equal, or adjacent at a rounding tie, or (with `quot_alts`, the oracle's
    quotients for G moved by its fp32 error bound) within the codes that the quotient
    range around the exact-G quotient rounds to."""
    diff = gpu != ora
    stats = dict(n=int(gpu.size), ties=0, g_window=0)
    if not diff.any():
        return stats
    g, o, q = gpu[diff].astype(np.int64), ora[diff].astype(np.int64), quot[diff]
    gv = oracle.e4m3_decode(g.astype(np.uint8))
    adjacent = ((g >> 7) == (o >> 7)) & (np.abs((g & 0x7F) - (o & 0x7F)) == 1)
    mid = 0.5 * (np.abs(gv) + np.abs(oracle.e4m3_decode(o.astype(np.uint8))))
    near = np.abs(np.abs(q) - mid) <= rel * np.abs(q) + 2.0 ** -12
    floor = (g == 1) & (o == 1)
    ok = (adjacent & near) | floor
    stats["ties"] = int(ok.sum())
    if len(quot_alts):
        qs = np.stack([q] + [a[diff] for a in quot_alts])
        lo = oracle.e4m3_decode(oracle.e4m3_encode(np.clip(qs.min(axis=0), -448, 448)))
        hi = oracle.e4m3_decode(oracle.e4m3_encode(np.clip(qs.max(axis=0), -448, 448)))
        win = ~ok & (gv >= lo) & (gv <= hi)
        stats["g_window"] = int(win.sum())
        ok |= win
    if not ok.all():
        i = np.flatnonzero(~ok)[:5]
        raise AssertionError(f"{name}: {int((~ok).sum())} codes differ beyond ties, e.g. "
                             f"{list(zip(g[i].tolist(), o[i].tolist(), q[i].tolist()))}")
    return stats


def check_ring(gpu, ora, slot, name):
    clr = (slot + 1) % 4
    assert gpu[clr] == 0.0 and ora[clr] == 0.0, f"{name}: slot {clr} not cleared"
    np.testing.assert_allclose(gpu[slot], ora[slot], rtol=1e-5, err_msg=f"{name} slot {slot}")


MODES = {"m": (False, True), "w": (True, False), "wm": (True, True)}


@pytest.mark.parametrize("shape", [(77, 328, 200), (256, 264, 520), (1, 8, 8), (512, 4096, 4096),
                                   (512, 14336, 4096)],
                         ids=lambda s: "x".join(map(str, s)))
@pytest.mark.parametrize("mode", list(MODES))
def test_fp8_three_steps_from_cold_start(mode, shape):
    w8, m8 = MODES[mode]
    T, d_in, d_out = shape
    _say(f"fp8 {mode} T={T} d_in={d_in} d_out={d_out}")
    dev = torch.device("cuda:0")
    W0 = synth.gaussian((d_out, d_in), 0.02, 9901)
    if w8:
        # fp8 weights start from W0 encoded with its own amax as the scale (slots (t-2)%4 and
        # (t-1)%4 of step 1 hold that amax)
        a = np.float32(np.abs(oracle.bf16_bits_to_f64(bits(W0))).max())
        ring = np.zeros(4, np.float32)
        ring[3] = ring[0] = a
        Wc = oracle.e4m3_encode(np.clip(oracle.bf16_bits_to_f64(bits(W0)).astype(np.float32) / (a / np.float32(448)),
                                        -448, 448))
        W, w_ring = fp8_tensor(Wc), torch.from_numpy(ring).to(dev)
    else:
        W, w_ring = W0.to(dev), None
    if m8:
        m = fp8_tensor(np.zeros((d_out, d_in), np.uint8))
        v = fp8_tensor(np.zeros((d_out, d_in), np.uint8))
        m_ring = torch.zeros(4, dtype=torch.float32, device=dev)
        v_ring = torch.zeros(4, dtype=torch.float32, device=dev)
    else:
        m = torch.zeros((d_out, d_in), dtype=torch.bfloat16, device=dev)
        v = torch.zeros((d_out, d_in), dtype=torch.bfloat16, device=dev)
        m_ring = v_ring = None
    host = lambda t, is8: codes(t) if is8 else bits(t)
    for step in (1, 2, 3):
        X = synth.gaussian((T, d_in), 1.0, 9910 + step, device=dev)
        dY = synth.gaussian((T, d_out), 1e-3, 9920 + step, device=dev)
        G = oracle.wgrad(bits(X), bits(dY))
        EG = gemm_error_bound(bits(X), bits(dY))
        state = (host(W, w8), host(m, m8), host(v, m8))
        rings = dict(w_ring=bits(w_ring) if w8 else None, m_ring=bits(m_ring) if m8 else None,
                     v_ring=bits(v_ring) if m8 else None)
        ora, lo, hi = (oracle.adamw_fp8(G + d, *state, w_fp8=w8, m_fp8=m8, step=step, **rings, **HP)
                       for d in (0.0, -EG, EG))
        if w8:
            forge.forge_linear_step_wfp8(X, dY, W, w_ring, m, v, m_ring, v_ring, step=step, **HP)
        else:
            forge.forge_linear_step(X, dY, W, m, v, m_ring, v_ring, step=step, **HP)
        torch.cuda.synchronize()
        slot = step % 4
        out = {}
        if w8:
            out["W"] = check_e4m3(codes(W), ora["W"], ora["qw"], "W", quot_alts=(lo["qw"], hi["qw"]))
            check_ring(bits(w_ring), ora["w_ring"], slot, "w_ring")
        else:
            out["W"] = check_weight(bits(W), ora["W"])
        if m8:
            out["m"] = check_e4m3(codes(m), ora["m"], ora["qm"], "m", quot_alts=(lo["qm"], hi["qm"]))
            out["v"] = check_e4m3(codes(v), ora["v"], ora["qv"], "sqrt(v)", quot_alts=(lo["qv"], hi["qv"]))
            check_ring(bits(m_ring), ora["m_ring"], slot, "m_ring")
            check_ring(bits(v_ring), ora["v_ring"], slot, "v_ring")
        else:
            wm, wv = moment_windows(dict(ora, G=G, EG=EG), HP)
            out["m"] = check_moment(bits(m), ora["m"], ora["m64"], "bf16", "m", window=wm)
            out["v"] = check_moment(bits(v), ora["v"], ora["v64"], "bf16", "v", window=wv)
        _say(f"step {step}: {out}")


def test_fp8_grouped_and_backward_equal_single_calls():
    """fp8 moments in a grouped launch and through the layer-level backward: bit-identical
    to single forge_linear_step calls (each matrix with its own rings)."""
    dev = torch.device("cuda:0")
    T, d_in = 96, 264
    X = synth.gaussian((T, d_in), 1.0, 9931, device=dev)
    mats_a, mats_b = [], []
    for i, d_out in enumerate((264, 72, 136)):
        dY = synth.gaussian((T, d_out), 1e-3, 9940 + i, device=dev)
        W = synth.gaussian((d_out, d_in), 0.02, 9950 + i, device=dev)
        m = fp8_tensor(oracle.e4m3_encode(np.full((d_out, d_in), 0.5, np.float32)))
        v = fp8_tensor(oracle.e4m3_encode(np.full((d_out, d_in), 0.25, np.float32)))
        ring = torch.tensor([0.0, 1e-3 * 448, 0.0, 1e-3 * 448], dtype=torch.float32, device=dev)
        st = (W, m, v, ring, ring.clone())
        mats_a.append((X, dY) + tuple(t.clone() for t in st))
        mats_b.append((X, dY) + tuple(t.clone() for t in st))
    dX = torch.empty((T, d_in), dtype=torch.bfloat16, device=dev)
    forge.forge_linear_backward_grouped(mats_a, dX=dX, step=5, **HP)
    for mt in mats_b:
        forge.forge_linear_step(*mt, step=5, **HP)
    torch.cuda.synchronize()
    for a, b in zip(mats_a, mats_b):
        for x, y in zip(a[2:], b[2:]):
            assert torch.equal(x.contiguous().view(torch.uint8), y.contiguous().view(torch.uint8))
