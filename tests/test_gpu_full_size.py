"""GPU parity at full and maximum sizes, on sampled outputs the oracle computes one by one.

Def. 1 / Prop. 1: the step is tile-local.  Row p of the new W, m and v depends only on
column p of dY, on X, and on row p of the old state (and column q only on column q of
X).  So the oracle run on a subset of rows (or columns) gives exactly the values the
full problem has there, and a full-size GPU result can be checked on a sample.

* The Llama-3.1-8B sweep (225 matrices, T=512, bf16 moments) is stepped exactly as the
  benchmark times it: ``forge_linear_step_grouped`` per backward-order group of matrices
  (``synth.launch_groups``), back to back on one stream.
* The largest legal operands: X or dY with just under 2^31 elements and a ragged token
  count, so the last token chunk runs past T at byte offsets beyond 2^32; and fp32 moments
  of 1.56 G elements (6.2 GB each), whose rows lie beyond the 4 GB a buffer offset reaches.
"""
import numpy as np
import pytest
import torch

import oracle
from compare import check_step
from gpu_util import Problem, bits, run_oracle
from paper_2606_22932_amd import forge, synth

pytestmark = pytest.mark.gpu

ROWS_PER_MATRIX = 8


def _say(*a):
    print(*a, flush=True)


def _sample(n, rng, k, tile=128):
    """k indices in [0, n): both ends, a tile boundary, and seeded random ones."""
    fixed = {0, n - 1} | ({tile - 1, tile} if n > tile else set())
    extra = rng.choice(n, size=max(0, k - len(fixed)), replace=False)
    return np.array(sorted(fixed | {int(i) for i in extra}), dtype=np.int64)


def test_sweep_sampled_rows_in_bench_configuration():
    wl = synth.WORKLOADS["sweep"]
    step = wl.steps[0]
    device = torch.device("cuda:0")
    rng = np.random.default_rng(2606)
    tensors, expected = [], []
    for mat in wl.matrices:
        X, dY = synth.activations(wl.T, mat, wl, step, device=device)
        W = synth.weight(mat, wl, device=device)
        m, v = synth.warm_moments(mat, wl, device=device, dtype=torch.bfloat16)
        rows = _sample(mat.d_out, rng, ROWS_PER_MATRIX)
        r = torch.from_numpy(rows).to(device)
        p = Problem(bits(X), bits(dY.index_select(1, r)), bits(W.index_select(0, r)),
                    bits(m.index_select(0, r)), bits(v.index_select(0, r)), "bf16", hp=dict(wl.hyper))
        expected.append((mat, r, p, run_oracle(p, step)))
        tensors.append((X, dY, W, m, v))
    groups = synth.launch_groups(wl)
    _say(f"sweep: {len(tensors)} matrices generated; one fused step in {len(groups)} grouped launches")
    for g in groups:
        forge.forge_linear_step_grouped([tensors[i] for i in g], step=step, **wl.hyper)
    torch.cuda.synchronize()
    n = 0
    for (X, dY, W, m, v), (mat, r, p, ora) in zip(tensors, expected):
        gpu = dict(W=bits(W.index_select(0, r)), m=bits(m.index_select(0, r)), v=bits(v.index_select(0, r)))
        try:
            check_step(gpu, ora, "bf16", hp=p.hp)
        except AssertionError as e:
            raise AssertionError(f"{mat.name} rows {r.tolist()}: {e}") from None
        n += gpu["W"].size
    _say(f"sweep: {n} sampled elements of W, m, v checked")


# (T, d_in, d_out): X (then dY) with just under 2^31 elements, T ragged against the
# 32-token chunk; chunk 1 holds one token row and its other rows lie past 2^32 bytes.
D_MAX = 65075256          # 33 * D_MAX = 2147483448 < 2^31 - 1, and a multiple of 8
MAX_SHAPES = [(33, D_MAX, 8, "bf16"), (33, D_MAX, 8, "i8"), (33, D_MAX, 8, "i8r64"), (33, 8, D_MAX, "bf16"),
              (33, D_MAX, 24, "f32")]


@pytest.mark.parametrize("T,d_in,d_out,moment", MAX_SHAPES,
                         ids=["X-2^31-bf16", "X-2^31-i8", "X-2^31-i8r64", "dY-2^31-bf16", "X-2^31-f32-6GB-moments"])
def test_maximum_operand_size(T, d_in, d_out, moment):
    _say(f"max size T={T} d_in={d_in} d_out={d_out} {moment}")
    device = torch.device("cuda:0")
    hp = dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.1)
    base = 7000
    X = synth.gaussian((T, d_in), 1.0, base + 1, device=device)
    dY = synth.gaussian((T, d_out), 1e-3, base + 11, device=device)
    W = synth.gaussian((d_out, d_in), 0.02, base + 2, device=device)
    mat = synth.Matrix("max", d_out, d_in, base)
    wl = synth.WORKLOADS["o_proj"]
    if moment in ("i8", "i8r64"):
        m, v, ms, vs = synth.random_i8_state(mat, wl, device=device, layout="col256" if moment == "i8" else "row64")
    else:
        m, v = synth.warm_moments(mat, wl, device=device,
                                  dtype=torch.float32 if moment == "f32" else torch.bfloat16)
        ms = vs = None
    rng = np.random.default_rng(33)
    if moment == "i8r64":
        # sample whole 64-column blocks (a block's scale depends on all of its columns); the
        # last block holds the 56 columns of the ragged tail
        nb = (d_in + 63) // 64
        blocks = _sample(nb, rng, 8, tile=2)
        cols = torch.from_numpy(np.concatenate([np.arange(64 * b, min(64 * b + 64, d_in)) for b in blocks])).to(device)
        bsel = torch.from_numpy(blocks).to(device)
        sel = lambda t: t.index_select(1, cols)
        p = Problem(bits(sel(X)), bits(dY), bits(sel(W)), bits(sel(m)), bits(sel(v)), moment,
                    bits(ms.index_select(1, bsel)), bits(vs.index_select(1, bsel)), hp=dict(hp))
    elif d_in > d_out:
        # sample columns: X[:, cols], W/m/v[:, cols] (int8 scales are per column as well)
        cols = torch.from_numpy(_sample(d_in, rng, 64)).to(device)
        sel = lambda t: t.index_select(1, cols)
        p = Problem(bits(sel(X)), bits(dY), bits(sel(W)), bits(sel(m)), bits(sel(v)), moment,
                    bits(sel(ms)) if ms is not None else None, bits(sel(vs)) if vs is not None else None,
                    hp=dict(hp))
    else:
        rows = torch.from_numpy(_sample(d_out, rng, 64)).to(device)
        sel = lambda t: t.index_select(0, rows)
        p = Problem(bits(X), bits(dY.index_select(1, rows)), bits(sel(W)), bits(sel(m)), bits(sel(v)),
                    moment, hp=dict(hp))
    ora = run_oracle(p, 100)
    forge.forge_linear_step(X, dY, W, m, v, ms, vs, step=100, **hp)
    torch.cuda.synchronize()
    gpu = dict(W=bits(sel(W)), m=bits(sel(m)), v=bits(sel(v)))
    if moment == "i8r64":
        gpu.update(m_scale=bits(ms.index_select(1, bsel)), v_scale=bits(vs.index_select(1, bsel)))
    elif ms is not None:
        gpu.update(m_scale=bits(sel(ms)), v_scale=bits(sel(vs)))
    _say(check_step(gpu, ora, moment, hp=p.hp))


# ----------------------------------------------------------------------------- layer-level backward

def _dx_rows_ok(got_rows, dY_rows, Ws, what):
    """Sampled token rows of dX against the oracle: row t of dX depends only on row t of
    each dY (and on the whole W), so the oracle on those rows gives the exact values."""
    from test_gpu_backward import check_dx
    try:
        return check_dx(got_rows, list(zip(dY_rows, Ws)))
    except AssertionError as e:
        raise AssertionError(f"{what}: {e}") from None


def test_backward_one_layer_and_lm_head_sampled_rows():
    """The backward of lm_head and of the last decoder layer of the sweep at T = 512, in
    its grouping ([down], [gate, up], [o], [q, k, v]): dX sampled on 8 token rows, the
    state sampled on 8 rows of each weight."""
    wl = synth.WORKLOADS["sweep"]
    step = wl.steps[0]
    device = torch.device("cuda:0")
    rng = np.random.default_rng(2607)
    groups = synth.launch_groups(wl)[:5]             # lm_head, then layer 31's four groups
    t_rows = _sample(wl.T, rng, 8)
    tr = torch.from_numpy(t_rows).to(device)
    for g in groups:
        tensors, host = [], []
        for i in g:
            mat = wl.matrices[i]
            X, dY = synth.activations(wl.T, mat, wl, step, device=device)
            W = synth.weight(mat, wl, device=device)
            m, v = synth.warm_moments(mat, wl, device=device, dtype=torch.bfloat16)
            rows = torch.from_numpy(_sample(mat.d_out, rng, ROWS_PER_MATRIX)).to(device)
            p = Problem(bits(X), bits(dY.index_select(1, rows)), bits(W.index_select(0, rows)),
                        bits(m.index_select(0, rows)), bits(v.index_select(0, rows)), "bf16", hp=dict(wl.hyper))
            host.append((mat, rows, p, run_oracle(p, step), bits(dY.index_select(0, tr)), bits(W)))
            tensors.append((X, dY, W, m, v))
        names = [h[0].name for h in host]
        _say(f"backward group {names}")
        dX = torch.empty((wl.T, tensors[0][0].shape[1]), dtype=torch.bfloat16, device=device)
        forge.forge_linear_backward_grouped(tensors, dX=dX, step=step, **wl.hyper)
        torch.cuda.synchronize()
        _say(_dx_rows_ok(bits(dX.index_select(0, tr)), [h[4] for h in host], [h[5] for h in host], names))
        for (X, dY, W, m, v), (mat, rows, p, ora, _, _) in zip(tensors, host):
            gpu = dict(W=bits(W.index_select(0, rows)), m=bits(m.index_select(0, rows)),
                       v=bits(v.index_select(0, rows)))
            check_step(gpu, ora, "bf16", hp=p.hp)


# (T, d_in, d_out): dY (then dX and W) with just under 2^31 elements.  W is zero except on
# 64 sampled rows, so that dX = dY[:, rows] W[rows, :] exactly and the oracle stays cheap
# while the kernel still runs its whole K loop.
DX_MAX_SHAPES = [(33, 8, D_MAX), (33, D_MAX, 8)]


@pytest.mark.parametrize("T,d_in,d_out", DX_MAX_SHAPES, ids=["dY-2^31", "dX-2^31"])
def test_input_grad_maximum_operand_size(T, d_in, d_out):
    _say(f"input_grad max size T={T} d_in={d_in} d_out={d_out}")
    device = torch.device("cuda:0")
    rng = np.random.default_rng(34)
    dY = synth.gaussian((T, d_out), 1e-3, 7101, device=device)
    W = synth.gaussian((d_out, d_in), 0.02, 7102, device=device)
    rows = torch.from_numpy(_sample(d_out, rng, 8)).to(device)
    if d_out > 64:
        keep = torch.zeros(d_out, dtype=torch.bool, device=device)
        keep[rows] = True
        W[~keep] = 0
    dX = torch.full((T, d_in), float("nan"), dtype=torch.bfloat16, device=device)
    forge.forge_input_grad(dY, W, dX)
    torch.cuda.synchronize()
    from test_gpu_backward import check_dx
    if d_in > 64:
        cols = torch.from_numpy(_sample(d_in, rng, 64)).to(device)
        got = bits(dX.index_select(1, cols))
        _say(check_dx(got, [(bits(dY), bits(W.index_select(1, cols)))]))
        assert not torch.isnan(dX).any()
    else:
        _say(check_dx(bits(dX), [(bits(dY.index_select(1, rows)), bits(W.index_select(0, rows)))]))
