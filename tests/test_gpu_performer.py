"""Parity of the Performer (FAVOR+) attention variant (the backbone Sec. 6
names) between the HIP path and the oracle, at the main and large workloads'
shapes in bf16 and the small workload's in fp32.

Weights are N(0, 0.05) with E, P scaled by 6 and Wq, Wk by 8, so that queries
and keys are large enough for the attention to be peaked (a maximum weight of
0.67-0.93 over 8 keys, against 1/8 for uniform); the feature projection is the
seeded orthogonal random features of synth.performer_features."""
import numpy as np
import pytest
import torch

import oracle as O
import synth
from gpu_helpers import check_parity, oracle_mode, to_dev, workload_cfg

pytestmark = pytest.mark.gpu


def _model(shape, dtype, flat, omega, **kw):
    import paper_2203_16114_amd as P
    m = P.TraceModel(**shape, dtype=dtype, attention="performer", **kw)
    m.init_weights(0, 0.02, flat)
    m.set_features(omega)
    return m


def _peaked_flat(cfg, seed):
    flat = O.init_flat(cfg, seed, 0.05)
    p = O.unflatten(flat, cfg)
    p["E"] *= 6
    p["P"] *= 6
    p["Wq"] *= 8
    p["Wk"] *= 8
    return O.flatten(p, cfg, np.float32)


@pytest.mark.parametrize("wid,dtype", [(3, "bf16"), (5, "bf16"), (2, "fp32"), (4, "bf16")])
def test_performer_forward_matches_oracle(wid, dtype):
    shape, _ = workload_cfg(wid)
    cfg = O.Config(**shape, attention="performer")
    flat = _peaked_flat(cfg, 0x9E4F + wid)
    omega = synth.performer_features(0x0FE4 + wid, cfg.m, cfg.dh)
    W = shape["W"]
    B, L = 192, W + 300
    streams, _ = synth.workload_streams(wid, L=L, B=B)
    m = _model(shape, dtype, flat, omega, max_windows=1 << 16, max_keep=B)
    s = to_dev(streams)
    b, i = synth.sample_positions(7 + wid, B, L, W, 256)
    ref = O.forward(flat, cfg, *O.windows_at(streams, b, i, W), mode=oracle_mode(dtype), features=omega)
    # wide tiles (a launch filling the chip), small tiles, and the kept variant
    n_steps = L - W
    big = m.forward_bits(s, W, n_steps, logits=True)
    idx = torch.from_numpy(b * n_steps + (i - W)).cuda()
    check_parity(dtype, big["logits"][idx].cpu().numpy(), big["bits"][idx].cpu().numpy(), ref)
    sub = slice(0, 32)
    for lo in range(0, 32, 8):
        p0 = int(i[lo])
        one = m.forward_bits(s, p0, 1, logits=True, keep=(lo == 8))
        zz = one["logits"][torch.from_numpy(b[lo:lo + 8]).cuda()].cpu().numpy()
        zr = big["logits"][torch.from_numpy(b[lo:lo + 8] * n_steps + (p0 - W)).cuda()].cpu().numpy()
        # the same windows in a one-step launch: the same kernel, bit for bit
        assert np.array_equal(zz.view(np.uint32), zr.view(np.uint32))
    # the weights really depart from uniform attention (1/T on every key)
    kept = O.forward(flat, cfg, *O.windows_at(streams, b[sub], i[sub], W), mode=oracle_mode(dtype), keep=True,
                     features=omega)
    last = kept["A"][:, :, -1, :]                    # [n][head][key] of the last query row
    assert np.mean(np.max(last, axis=-1)) > 4.0 / cfg.T, np.mean(np.max(last, axis=-1))


def test_performer_errors():
    import paper_2203_16114_amd as P
    shape, _ = workload_cfg(4)
    cfg = O.Config(**shape, attention="performer")
    m = P.TraceModel(**shape, dtype="bf16", attention="performer", max_keep=16)
    m.init_weights(3)
    s = to_dev(synth.random_streams(1, 16, 80))
    with pytest.raises(P.TraceError) as ei:
        m.forward_bits(s, 32, 4)
    assert ei.value.code == P.TRACE_ESTATE                      # features not set
    with pytest.raises(P.TraceError) as ei:
        m.set_features(np.zeros((cfg.m, cfg.dh + 1), np.float32))
    assert ei.value.code == P.TRACE_EINVAL
    m.set_features(synth.performer_features(1, cfg.m, cfg.dh))
    m.forward_bits(s, 32, 1, keep=True)
    with pytest.raises(P.TraceError) as ei:
        m.adapt_step()
    assert ei.value.code == P.TRACE_EUNSUPPORTED                # forward only
    soft = P.TraceModel(**shape, dtype="bf16")
    with pytest.raises(P.TraceError) as ei:
        soft.set_features(synth.performer_features(1, cfg.m, cfg.dh))
    assert ei.value.code == P.TRACE_EINVAL
