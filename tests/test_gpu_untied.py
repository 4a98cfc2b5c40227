"""The deep-FFN variant of Sec. 6.3: each of the k repeats of Eq. 3 with its
own W1, W2 (trace_config.untied_ffn).  Forward, gradient and Adam step
against the oracle with the same option, on both attention kernels."""
import numpy as np
import pytest

import oracle as O
import synth
from gpu_helpers import check_parity, to_dev

pytestmark = pytest.mark.gpu

SHAPE = dict(W=32, e=32, g=4, H=4, F=512, k=2)
SHAPE8 = dict(W=64, e=32, g=8, H=8, F=256, k=3)


def _model(shape, dtype, seed, **kw):
    import paper_2203_16114_amd as P
    m = P.TraceModel(**shape, dtype=dtype, untied_ffn=True, **kw)
    m.init_weights(seed)
    return m


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("shape,n_steps", [(SHAPE, 168), (SHAPE8, 128)])
def test_untied_forward_matches_oracle(dtype, shape, n_steps):
    """n_steps = 128 at 64-window tiles runs the shared-group attention kernel
    (bf16), 168 the token kernel."""
    W = shape["W"]
    streams = synth.random_streams(41, 12, W + n_steps + 1)
    m = _model(shape, dtype, 9, max_windows=1 << 14)
    out = m.forward_bits(to_dev(streams), W, n_steps, logits=True)
    cfg = O.Config(**shape, untied=True)
    w, y = O.all_windows(streams, W, W, n_steps)
    ref = O.forward(O.init_flat(cfg, 9), cfg, w, y, mode="fp64" if dtype == "fp32" else "bf16")
    check_parity(dtype, out["logits"].cpu().numpy(), out["bits"].cpu().numpy(), ref)


@pytest.mark.parametrize("dtype,B", [("fp32", 256), ("bf16", 300)])
def test_untied_gradient_and_adam_step_match_oracle(dtype, B):
    streams = synth.random_streams(31, B, 100)
    m = _model(SHAPE, dtype, 0x1234, max_keep=B)
    th0 = m.get_state()[0]
    m.forward_bits(to_dev(streams), 50, 1, keep=True)
    m.adapt_step()
    g = m.grads()
    th1 = m.get_state()[0]
    cfg = O.Config(**SHAPE, untied=True)
    flat = O.init_flat(cfg, 0x1234)
    w, y = O.windows_at(streams, np.arange(B), np.full(B, 50), 32)
    _, ref = O.forward_backward(flat, cfg, w, y, mode="fp64" if dtype == "fp32" else "bf16")
    gp = O.unflatten(g, cfg)
    for name, _ in O.param_layout(cfg):
        a = gp[name].astype(np.float64)
        b = np.asarray(ref[name], np.float64)
        if dtype == "fp32":
            scale = np.max(np.abs(b))
            assert np.all(np.abs(a - b) <= 1e-4 * np.abs(b) + 1e-5 * scale), name
        else:
            assert np.linalg.norm(a - b) <= 1e-2 * max(np.linalg.norm(b), 1e-30), name
    # the per-repeat blocks differ (the repeats are not interchangeable)
    assert not np.allclose(gp["W1"][0], gp["W1"][1])
    # one Adam step on the oracle's own gradient
    opt = O.Adam(flat.size, cfg)
    flat1 = opt.step(flat, O.flatten(ref, cfg, np.float32))
    d_gpu, d_ref = th1.astype(np.float64) - th0, flat1.astype(np.float64) - flat
    assert np.linalg.norm(d_gpu - d_ref) <= 1e-3 * np.linalg.norm(d_ref)
