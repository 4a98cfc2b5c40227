"""trace_forward_bits_noalloc: the forward for callers that cannot allocate,
with its attention -> FFN hand-off in the library's fixed device array.  Same
launches as trace_forward_bits, so its results must equal that entry point's
bit for bit, on consecutive calls of different sizes (the array keeps the
previous call's contents)."""
import numpy as np
import pytest
import torch

import synth
from gpu_helpers import make_model, to_dev

pytestmark = pytest.mark.gpu

SCRATCH_BYTES = 32 << 20


def _both(m, s, pos0, n_steps, **kw):
    a = m.forward_bits(s, pos0, n_steps, logits=True, step_ce=True, **kw)
    b = m.forward_bits(s, pos0, n_steps, logits=True, step_ce=True, noalloc=True, **kw)
    torch.cuda.synchronize()
    return a, b


def _equal(a, b):
    for k in ("bits", "logits", "step_ce"):
        assert torch.equal(a[k], b[k]), k


@pytest.mark.parametrize("shape,dtype", [(dict(W=64, e=32, g=8, H=8, F=1024, k=3), "bf16"),
                                         (dict(W=32, e=32, g=4, H=4, F=512, k=2), "fp32"),
                                         (dict(W=64, e=64, g=8, H=8, F=2048, k=3), "bf16")])
def test_noalloc_forward_equals_forward_on_two_calls(shape, dtype):
    d = shape["e"] * shape["g"]
    cap = SCRATCH_BYTES // (4 * d)
    W = shape["W"]
    m = make_model(shape, dtype, seed=31)
    # first call: the largest batch the array holds (whole 64-window tiles per stream)
    B1, S1 = cap // 256, 256
    st = synth.random_streams(41, B1, W + S1 + 1)
    a, b = _both(m, to_dev(st), W, S1)
    _equal(a, b)
    # second call: smaller and ragged, after the first left its values in the array
    st2 = synth.random_streams(42, 7, W + 40)
    a2, b2 = _both(m, to_dev(st2), W + 3, 33)
    _equal(a2, b2)
    a3, b3 = _both(m, to_dev(st2), W + 1, 5, token_attn=True)
    _equal(a3, b3)


def test_noalloc_rejects_batches_beyond_the_array():
    import paper_2203_16114_amd as P
    shape = dict(W=64, e=32, g=8, H=8, F=1024, k=3)
    m = make_model(shape, "bf16", seed=3)
    cap = SCRATCH_BYTES // (4 * 256)
    st = to_dev(synth.random_streams(5, 2, 64 + cap // 2 + 2))
    with pytest.raises(P.TraceError) as ei:
        m.forward_bits(st, 64, cap // 2 + 1, noalloc=True)
    assert ei.value.code == P.TRACE_EINVAL
    # the model and the array are still usable
    a, b = _both(m, st, 64, 64)
    _equal(a, b)
