"""The fused paths allocate no device memory: a call leaves torch's allocator and the
device's free memory where they were (the library takes caller-owned buffers and keeps no
workspace; the kernels need none)."""
import gc

import pytest
import torch

from paper_2606_22932_amd import forge, synth

pytestmark = pytest.mark.gpu

HP = dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.1)


def _mats(moment, n, T=200, d_in=520, d_out=392, seed=900):
    dev = "cuda"
    X = synth.gaussian((T, d_in), 1.0, seed, device=dev)
    out = []
    for i in range(n):
        dY = synth.gaussian((T, d_out), 1e-3, seed + 10 + i, device=dev)
        W = synth.gaussian((d_out, d_in), 0.02, seed + 20 + i, device=dev)
        if moment == "bf16":
            m = synth.gaussian((d_out, d_in), 1e-4, seed + 30 + i, device=dev)
            v = synth.gaussian((d_out, d_in), 1e-6, seed + 40 + i, device=dev, absolute=True)
            out.append((X, dY, W, m, v, None, None))
        else:
            mat = synth.Matrix("m", d_out, d_in, seed + i)
            m, v, ms, vs = synth.random_i8_state(mat, synth.WORKLOADS["o_proj"], device=dev,
                                                 layout="col256" if moment == "i8" else "row64")
            out.append((X, dY, W, m, v, ms, vs))
    return X, out


def _snapshot():
    torch.cuda.synchronize()
    return torch.cuda.memory_allocated(), torch.cuda.memory_reserved(), torch.cuda.mem_get_info()[0]


class _no_gc:
    """Collect garbage first and keep the collector off inside the measured window, so that
    tensors freed by an earlier test cannot lower the figures during the call."""
    def __enter__(self):
        gc.collect()
        gc.disable()

    def __exit__(self, *exc):
        gc.enable()


@pytest.mark.parametrize("moment", ["bf16", "i8", "i8r64"])
def test_fused_step_grouped_and_backward_allocate_nothing(moment):
    X, mats = _mats(moment, 3)
    dX = torch.empty_like(X)

    def calls(step):
        forge.forge_linear_step(*mats[0], step=step, **HP)
        forge.forge_linear_step_grouped(mats, step=step, **HP)
        forge.forge_linear_backward(*mats[1], dX=dX, step=step, **HP)
        forge.forge_linear_backward_grouped(mats, dX=dX, step=step, **HP)

    calls(1)                       # code objects loaded, first launches done
    with _no_gc():
        before = _snapshot()
        for t in range(2, 5):
            calls(t)
        after = _snapshot()
    print(f"{moment}: allocated/reserved/free before {before}, after {after}", flush=True)
    assert after == before
