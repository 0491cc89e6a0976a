"""forge_linear_step_unfused_noalloc: the two-kernel step with G in the library's fixed
device buffer instead of a caller workspace.

Checked against forge_linear_step_unfused with a torch-allocated workspace on the same
inputs: W, m, v (and the int8 scales) must be bit-identical (both run the same GEMM and
optimizer kernels on the same G), on two calls in a row with the second smaller than the
first, and at the buffer's maximum size.  The call must leave torch's allocator and the
device's free memory unchanged, and a gradient larger than the buffer is refused.
"""
import gc

import pytest
import torch

from gpu_util import dev, make_problem
from paper_2606_22932_amd import forge

pytestmark = pytest.mark.gpu

GRAD_BYTES = {"bf16": 2, "f32": 4}


def _say(*a):
    print(*a, flush=True)


def _state(p):
    t = [dev(a) for a in (p.W, p.m, p.v)]
    t += [dev(p.m_scale), dev(p.v_scale)] if p.m_scale is not None else [None, None]
    return t


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


@pytest.fixture(scope="module", autouse=True)
def buffer_set_up():
    """The first call on a device looks up the buffer's address; the HIP runtime may load
    the library's code object that holds the buffer at that moment (once per device, held
    until the process ends).  Every call measured below comes after it."""
    p = make_problem(8, 8, 8, "bf16", seed=59)
    X, dY = dev(p.X), dev(p.dY)
    W, m, v, _, _ = _state(p)
    forge.forge_linear_step_unfused_noalloc(X, dY, W, m, v, grad_dtype="bf16", step=1, **p.hp)
    torch.cuda.synchronize()


def _compare(p, grad, step):
    X, dY = dev(p.X), dev(p.dY)
    a, b = _state(p), _state(p)
    G = torch.empty(p.W.shape, dtype=torch.bfloat16 if grad == "bf16" else torch.float32, device="cuda")
    forge.forge_linear_step_unfused(X, dY, *a, G_ws=G, step=step, **p.hp)
    with _no_gc():
        before = _snapshot()
        forge.forge_linear_step_unfused_noalloc(X, dY, *b, grad_dtype=grad, step=step, **p.hp)
        after = _snapshot()
    assert after == before, f"allocation seen: {before} -> {after}"
    for x, y, name in zip(a, b, ("W", "m", "v", "m_scale", "v_scale")):
        if x is not None:
            assert torch.equal(x.view(torch.uint8), y.view(torch.uint8)), f"{name} differs"


@pytest.mark.parametrize("moment", ["f32", "bf16", "i8", "i8r64"])
@pytest.mark.parametrize("grad", ["bf16", "f32"])
def test_noalloc_equals_workspace_path_two_calls(moment, grad):
    # the second call is smaller: the buffer keeps the first call's G beyond its own range
    for i, shape in enumerate([(200, 1032, 776), (77, 328, 264)]):
        _say(f"noalloc {moment} grad={grad} call {i + 1}: T,d_in,d_out={shape}")
        p = make_problem(*shape, moment, seed=60 + i)
        _compare(p, grad, step=9 + i)


@pytest.mark.parametrize("grad", ["bf16", "f32"])
def test_noalloc_at_the_buffer_size_and_beyond(grad):
    d_out = 4096
    d_in = forge.FORGE_SCRATCH_BYTES // (GRAD_BYTES[grad] * d_out)     # exactly the buffer
    _say(f"noalloc at the limit: grad={grad} d_in={d_in} d_out={d_out}")
    p = make_problem(64, d_in, d_out, "bf16", seed=70)
    _compare(p, grad, step=3)
    # one more row of 8 columns does not fit: refused on the host, nothing launched
    q = make_problem(8, d_in + 8, d_out, "bf16", seed=71)
    X, dY = dev(q.X), dev(q.dY)
    W, m, v, _, _ = _state(q)
    W0 = W.clone()
    with pytest.raises(forge.ForgeError) as e:
        forge.forge_linear_step_unfused_noalloc(X, dY, W, m, v, grad_dtype=grad, step=1, **q.hp)
    assert e.value.name == "FORGE_ERR_SCRATCH_LIMIT"
    torch.cuda.synchronize()
    assert torch.equal(W, W0)
