"""The gated loop of Alg. 1 with the controller of Alg. 2 (trace_gated_run).

Its forwards run ahead over several steps at unchanged weights and the
controller walks their step cross-entropies.  That gives the decisions of a
loop of one-step forwards only if every window's code length is the same bit
for bit whatever launch it was computed in: the per-token attention kernel
(TRACE_TOKEN_ATTN) guarantees that, and these tests check it, then check that
the speculative run equals one-step loops step for step."""
import numpy as np
import pytest
import torch

import paper_2203_16114_amd as P
import synth
from gpu_helpers import make_model, to_dev, workload_cfg

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("wid,B", [(4, 4096), (5, 8192), (2, 512)])
def test_token_attention_is_launch_invariant(wid, B):
    shape, dtype = workload_cfg(wid)
    W = shape["W"]
    pos0, S = 3 * W + 5, 64
    streams, _ = synth.workload_streams(wid, L=pos0 + S + 1, B=B)
    s = to_dev(streams)
    m = make_model(shape, dtype, seed=0x600D + wid, max_windows=B * S, max_keep=B)
    many = m.forward_bits(s, pos0, S, step_ce=True, token_attn=True)
    bits = many["bits"].view(B, S)
    ce = many["step_ce"]
    for q in range(S):
        one = m.forward_bits(s, pos0 + q, 1, step_ce=True, keep=(q % 16 == 0))
        assert torch.equal(one["bits"], bits[:, q]), q
        assert torch.equal(one["step_ce"][0], ce[q]), q
    # a launch starting at another position and split into chunks
    m2 = make_model(shape, dtype, seed=0x600D + wid, max_windows=1000, max_keep=B)
    part = m2.forward_bits(s, pos0 + 7, S - 7, step_ce=True, token_attn=True)
    assert torch.equal(part["bits"].view(B, S - 7), bits[:, 7:])
    assert torch.equal(part["step_ce"], ce[7:])


def _one_step_loop(m, s, pos0, n_steps, t, delta):
    """The loop of Alg. 1 written out with one-step forwards: estimate, decide,
    and on an update the backward + Adam step on that batch."""
    ctl = P.Controller(t, delta)
    ce, dec = [], []
    for q in range(n_steps):
        out = m.forward_bits(s, pos0 + q, 1, step_ce=True, keep=True)
        e = float(out["step_ce"][0])
        d = ctl.decide(e)
        if d:
            m.adapt_step()
        ce.append(e)
        dec.append(d)
    return np.array(ce), np.array(dec, np.int32)


@pytest.mark.parametrize("delta,B,t", [(0.0, 4096, 16), (0.0, 512, 4)])
def test_speculative_gated_run_equals_the_one_step_loop(delta, B, t):
    """delta = 0 is Eq. 7 literally.  A model this close to its random start
    has step cross-entropies within a few thousandths of a bit of their
    running mean (8 bits) once it stops updating, so a margin of 0.05 bits is
    never crossed after the warm-up; with delta = 0 about half the steps are
    updated."""
    shape, dtype = workload_cfg(4)
    n = 320
    pos0 = 2048 - 160            # crosses the source switch at byte 2048
    streams, _ = synth.workload_streams(4, L=pos0 + n + 1, B=B)
    s = to_dev(streams)
    seed = 0x7ACE1004
    runs = {}
    for name, spec in (("spec64", 64), ("spec1", 1)):
        m = make_model(shape, dtype, seed, max_windows=B * 64, max_keep=B)
        ce, dec, nu = m.gated_run(s, pos0, n, P.MODE_GATED, t, delta, max_spec=spec)
        runs[name] = (ce, dec, nu, m.get_state())
    m = make_model(shape, dtype, seed, max_windows=B * 64, max_keep=B)
    ce1, dec1 = _one_step_loop(m, s, pos0, n, t, delta)
    runs["loop"] = (ce1, dec1, int(dec1.sum()), m.get_state())
    ref = runs["spec64"]
    assert ref[1][:t].sum() == t                     # warm-up
    post = int(ref[1][t:].sum())
    assert 0 < post < n - t, post                    # the controller decided both ways after warm-up
    for name in ("spec1", "loop"):
        ce, dec, nu, st = runs[name]
        assert np.array_equal(ce.view(np.uint64), ref[0].view(np.uint64)), name
        assert np.array_equal(dec, ref[1]) and nu == ref[2], name
        for a, b in zip(st[:3], ref[3][:3]):
            assert np.array_equal(a.view(np.uint32), b.view(np.uint32)), name
        assert st[3] == ref[3][3] == ref[2]


def test_gated_run_modes_never_and_always():
    shape, dtype = workload_cfg(4)
    B, n = 1024, 70
    streams, _ = synth.workload_streams(4, L=200 + n + 1, B=B)
    s = to_dev(streams)
    m = make_model(shape, dtype, 5, max_windows=B * 64, max_keep=B)
    ce0, dec0, nu0 = m.gated_run(s, 200, n, P.MODE_NEVER, max_spec=32)
    assert nu0 == 0 and not dec0.any()
    frozen = m.forward_bits(s, 200, n, step_ce=True, token_attn=True)["step_ce"].cpu().numpy()
    assert np.array_equal(ce0, frozen)
    ca, da, nua = m.gated_run(s, 200, n, P.MODE_ALWAYS)
    assert nua == n and da.all() and m.get_state()[3] == n
    m2 = make_model(shape, dtype, 5, max_windows=B * 64, max_keep=B)
    cb, db = _one_step_loop(m2, s, 200, n, 1, -1e30)      # the controller with delta = -inf: always
    assert np.array_equal(ca, cb)
    with pytest.raises(P.TraceError) as ei:
        make_model(shape, dtype, 5).gated_run(s, 200, 4, P.MODE_GATED)   # no max_keep
    assert ei.value.code == P.TRACE_EINVAL
