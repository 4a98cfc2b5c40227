"""Stacked layers (Sec. 6.3, Fig. 7): forward and gradient parity of the HIP
path with the oracle.  The lower layers run over every token row (their
attention over all T query rows, the projections and FFN as GEMMs on the
update's kernels); the top layer runs in the fused kernels with the lower
layers' output as its input rows."""
import numpy as np
import pytest
import torch

import oracle as O
import synth
from gpu_helpers import check_parity, oracle_mode, to_dev, workload_cfg

pytestmark = pytest.mark.gpu


def _model(shape, dtype, layers, seed, **kw):
    import paper_2203_16114_amd as P
    m = P.TraceModel(**shape, dtype=dtype, layers=layers, **kw)
    m.init_weights(seed)
    return m


@pytest.mark.parametrize("wid,dtype,layers", [(4, "bf16", 2), (4, "bf16", 3), (2, "fp32", 2), (1, "fp32", 3),
                                              (3, "bf16", 2), (5, "bf16", 2)])
def test_multilayer_forward_matches_oracle(wid, dtype, layers):
    shape, _ = workload_cfg(wid)
    cfg = O.Config(**shape, layers=layers)
    seed = 0x1A4E + wid
    W = shape["W"]
    B, L = 96, W + 200
    streams, _ = synth.workload_streams(wid, L=L, B=min(B, synth.WORKLOADS[wid].B))
    B = streams.shape[0]
    m = _model(shape, dtype, layers, seed, max_windows=4096)
    s = to_dev(streams)
    n_steps = L - W
    out = m.forward_bits(s, W, n_steps, logits=True)            # several chunks of 4096 windows
    flat = O.init_flat(cfg, seed)
    b, i = synth.sample_positions(11 + wid, B, L, W, 192)
    ref = O.forward(flat, cfg, *O.windows_at(streams, b, i, W), mode=oracle_mode(dtype))
    idx = torch.from_numpy(b * n_steps + (i - W)).cuda()
    check_parity(dtype, out["logits"][idx].cpu().numpy(), out["bits"][idx].cpu().numpy(), ref)
    # one step over a few streams: the same results bit for bit
    one = m.forward_bits(s[:7].contiguous(), W + 33, 1, logits=True)
    assert torch.equal(one["logits"], out["logits"][torch.arange(7, device="cuda") * n_steps + 33])


@pytest.mark.parametrize("dtype,use_pos,B", [("fp32", True, 256), ("fp32", False, 130), ("bf16", True, 300)])
def test_multilayer_gradient_and_adam_step_match_oracle(dtype, use_pos, B):
    shape, _ = workload_cfg(4)
    layers = 2
    cfg = O.Config(**shape, layers=layers, use_pos=use_pos)
    seed = 0x2B5F
    streams, _ = synth.workload_streams(4, L=400, B=B)
    pos = 300
    m = _model(shape, dtype, layers, seed, use_pos=use_pos, max_keep=B)
    m.forward_bits(to_dev(streams), pos, 1, keep=True)
    m.adapt_step()
    g = O.unflatten(m.grads(), cfg)
    th = m.get_state()[0]
    flat = O.init_flat(cfg, seed)
    w, y = O.windows_at(streams, np.arange(B), np.full(B, pos), cfg.W)
    _, ref = O.forward_backward(flat, cfg, w, y, mode=oracle_mode(dtype))
    for name, _ in O.param_layout(cfg):
        a = np.asarray(g[name], np.float64)
        r = np.asarray(ref[name], np.float64)
        if dtype == "fp32":
            scale = np.max(np.abs(r)) if r.size else 0.0
            assert np.all(np.abs(a - r) <= 1e-4 * np.abs(r) + 1e-5 * scale), (name, np.max(np.abs(a - r)), scale)
        else:
            rel = np.linalg.norm(a - r) / max(np.linalg.norm(r), 1e-30)
            assert rel <= 1e-2, (name, rel)
        if name in ("Wq", "Wk", "Wv", "Wo", "W1", "W2"):   # every layer's block gets its own gradient
            for l in range(layers):
                assert np.linalg.norm(r[l]) > 0 and np.linalg.norm(a[l]) > 0, (name, l)
    if not use_pos:
        assert np.all(g["P"] == 0)
    # Adam on the GPU's gradient, in the oracle: bit for bit
    opt = O.Adam(flat.size, cfg)
    assert np.array_equal(opt.step(flat, m.grads()).view(np.uint32), th.view(np.uint32))
    # the updated model's forward against the oracle's forward of the new master
    out = m.forward_bits(to_dev(streams), pos + 1, 20, logits=True)
    bb, ii = np.meshgrid(np.arange(B), pos + 1 + np.arange(20), indexing="ij")
    r2 = O.forward(th, cfg, *O.windows_at(streams, bb.ravel(), ii.ravel(), cfg.W), mode=oracle_mode(dtype))
    check_parity(dtype, out["logits"].cpu().numpy(), out["bits"].cpu().numpy(), r2)


def test_multilayer_errors():
    import paper_2203_16114_amd as P
    shape, _ = workload_cfg(4)
    with pytest.raises(P.TraceError) as ei:
        P.TraceModel(**shape, dtype="bf16", layers=2, attention="performer")
    assert ei.value.code == P.TRACE_EINVAL
    with pytest.raises(P.TraceError) as ei:
        P.TraceModel(**shape, dtype="bf16", layers=9)
    assert ei.value.code == P.TRACE_EINVAL
