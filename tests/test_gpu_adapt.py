"""Parity of the gated update (gradient, Adam step, controller-gated steps)
between the HIP path and the CPU oracle, plus determinism and checkpointing.

Stages: (1) the gradient of one step; (2) the parameter change of one Adam
step, by norm, because near-zero gradients can flip the sign of an
element's +-lr step; (3) teacher-forced gated steps: the oracle replays the
GPU's decisions and the code lengths are compared step by step."""
import numpy as np
import pytest
import torch

import oracle as O
import synth
from gpu_helpers import check_parity, make_model, ocfg, to_dev

pytestmark = pytest.mark.gpu

SMALL = dict(W=32, e=32, g=4, H=4, F=512, k=2)   # the model of the small and adaptation workloads
NAMES = [n for n, _ in O.param_layout(ocfg(**SMALL))]


def _grad_run(shape, dtype, seed, streams, pos, use_pos=True):
    B = streams.shape[0]
    m = make_model(shape, dtype, seed, max_keep=B, use_pos=use_pos)
    m.forward_bits(to_dev(streams), pos, 1, keep=True)
    m.adapt_step()
    g = m.grads()
    th = m.get_state()[0]
    cfg = ocfg(**shape, use_pos=use_pos)
    flat = O.init_flat(cfg, seed)
    w, y = O.windows_at(streams, np.arange(B), np.full(B, pos), cfg.W)
    return m, cfg, flat, g, th, w, y


@pytest.mark.parametrize("use_pos", [True, False])
def test_fp32_gradient_matches_oracle(use_pos):
    streams = synth.random_streams(31, 256, 100)
    m, cfg, flat, g, _, w, y = _grad_run(SMALL, "fp32", 0x1234, streams, 50, use_pos)
    _, ref = O.forward_backward(flat, cfg, w, y, mode="fp64")
    gp = O.unflatten(g, cfg)
    for name in NAMES:
        a = gp[name].astype(np.float64)
        b = np.asarray(ref[name], np.float64)
        scale = np.max(np.abs(b)) if b.size else 0.0
        err = np.max(np.abs(a - b)) if b.size else 0.0
        # fp32 sums over up to N*T = 2048 products: per element 1e-4 relative,
        # with a floor of 1e-5 of the tensor's largest entry for entries that
        # cancel to near zero
        assert np.all(np.abs(a - b) <= 1e-4 * np.abs(b) + 1e-5 * scale), (name, err, scale)
    if not use_pos:
        assert np.all(gp["P"] == 0)


@pytest.mark.parametrize("B", [512, 300])
def test_bf16_gradient_matches_emulating_oracle(B):
    """B = 300: the products over the kept windows end in a partial k tile
    (their operands stored as bf16 included)."""
    streams, _ = synth.workload_streams(4, L=600, B=B)
    m, cfg, flat, g, _, w, y = _grad_run(SMALL, "bf16", 0x4321, streams, 500)
    _, ref = O.forward_backward(flat, cfg, w, y, mode="bf16")
    gp = O.unflatten(g, cfg)
    for name in NAMES:
        a = gp[name].astype(np.float64).ravel()
        b = np.asarray(ref[name], np.float64).ravel()
        # same bf16 storage points on both sides; what differs is the fp32
        # summation order, which can move an activation across a bf16 rounding
        # boundary (2^-8 relative on that element)
        rel = np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-30)
        assert rel <= 1e-2, (name, rel)


# d = 256 shapes of the rank-one key/value path (k_attn_bwd_r1 with four columns per
# lane, k_dx_rank1, k_rank1_sums, the positional-table gradient from window sums):
# the main workload's token shape (T = 8, dh = 32) and a T = 4 one (dh = 64)
RANK1_SHAPES = {
    "T8-dh32": dict(W=64, e=32, g=8, H=8, F=512, k=2),
    "T4-dh64": dict(W=32, e=32, g=8, H=4, F=512, k=2),
}


@pytest.mark.parametrize("name", sorted(RANK1_SHAPES))
def test_bf16_gradient_rank_one_shapes_match_emulating_oracle(name):
    """B = 300 windows (partial tiles and a partial window group of 16)."""
    shape = RANK1_SHAPES[name]
    streams = synth.random_streams(0x77 + len(name), 300, shape["W"] + 40)
    m, cfg, flat, g, _, w, y = _grad_run(shape, "bf16", 0x5150, streams, shape["W"] + 17)
    _, ref = O.forward_backward(flat, cfg, w, y, mode="bf16")
    gp = O.unflatten(g, cfg)
    for pname, _ in O.param_layout(cfg):
        a = gp[pname].astype(np.float64).ravel()
        b = np.asarray(ref[pname], np.float64).ravel()
        rel = np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-30)
        assert rel <= 1e-2, (name, pname, rel)
        assert np.linalg.norm(b) > 0, (name, pname)


# the key/value weight-gradient kernel at the shapes above and at d = 512 (the
# large workload's token shape, T = 8, dh = 64)
KV_SHAPES = dict(RANK1_SHAPES, **{"T8-d512": dict(W=64, e=64, g=8, H=8, F=512, k=1)})


@pytest.mark.parametrize("name", sorted(KV_SHAPES))
def test_kv_weight_gradient_in_kernel_gather_is_bitwise_the_update_gather(name):
    """dWk, dWv of the last update recomputed by the kernel from token rows
    written by the update's gather (bit-exact vs the oracle's embed_group in
    test_gpu_forward.py) and with the rows gathered inside the kernel: the same
    bits, so the in-kernel byte-group indexing is the tested one (Sec. 4.2)."""
    shape = KV_SHAPES[name]
    B = 300
    streams = synth.random_streams(0x5A + len(name), B, shape["W"] + 40)
    m = make_model(shape, "bf16", 0x77, max_keep=B)
    m.forward_bits(to_dev(streams), shape["W"] + 11, 1, keep=True)
    m.adapt_step()
    a, b = m.debug_kv_wgrad()
    torch.cuda.synchronize()
    a = a.cpu().numpy()
    b = b.cpu().numpy()
    assert np.isfinite(a).all() and np.abs(a).max() > 0
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))


@pytest.mark.parametrize("name", sorted(RANK1_SHAPES))
def test_bf16_gradient_rank_one_tiny_batch_matches_emulating_oracle(name):
    """B = 5 windows: fewer than one 32-window tile of the key/value weight
    gradients (the rest of the tile has zero coefficients, its rows read clamped)."""
    shape = RANK1_SHAPES[name]
    streams = synth.random_streams(0x99 + len(name), 5, shape["W"] + 40)
    m, cfg, flat, g, _, w, y = _grad_run(shape, "bf16", 0x5151, streams, shape["W"] + 9)
    _, ref = O.forward_backward(flat, cfg, w, y, mode="bf16")
    gp = O.unflatten(g, cfg)
    for pname, _ in O.param_layout(cfg):
        a = gp[pname].astype(np.float64).ravel()
        b = np.asarray(ref[pname], np.float64).ravel()
        rel = np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-30)
        assert rel <= 1e-2, (name, pname, rel)
        assert np.linalg.norm(b) > 0, (name, pname)


@pytest.mark.parametrize("kind", ["skewed", "one_byte"])
def test_fp32_embedding_gradient_over_many_sort_blocks(kind):
    """1100 kept windows of 32 bytes: 35200 positions, several blocks of the
    counting sort with a ragged last one.  Skewed: most bytes are one value
    (a byte run cut into many pieces); one_byte: every position holds the same
    byte.  The E gradient matches the oracle's to the fp32 bar."""
    B, L, pos = 1100, 40, 36
    streams = synth.random_streams(77, B, L)
    if kind == "skewed":
        rng = np.random.default_rng(5)
        streams = np.where(rng.random(streams.shape) < 0.8, np.uint8(32), streams).astype(np.uint8)
    else:
        streams = np.full_like(streams, 101)
    m, cfg, flat, g, _, w, y = _grad_run(SMALL, "fp32", 0x5150, streams, pos)
    _, ref = O.forward_backward(flat, cfg, w, y, mode="fp64")
    a = O.unflatten(g, cfg)["E"].astype(np.float64)
    b = np.asarray(ref["E"], np.float64)
    scale = np.max(np.abs(b))
    # sums over up to 35200 rows of fp32 values in a different order than the
    # oracle's: 1e-4 relative with a floor of 1e-5 of the largest entry
    assert np.all(np.abs(a - b) <= 1e-4 * np.abs(b) + 1e-5 * scale), np.max(np.abs(a - b))
    used = np.zeros(256, bool)
    used[np.unique(w)] = True
    assert np.all(a[~used] == 0)


def test_fp32_adam_step_matches_oracle():
    streams = synth.random_streams(32, 128, 90)
    m, cfg, flat, g, th, w, y = _grad_run(SMALL, "fp32", 77, streams, 40)
    _, ref = O.forward_backward(flat, cfg, w, y, mode="fp64")
    opt = O.Adam(flat.size, cfg)
    th_ref = opt.step(flat, O.flatten(ref, cfg, np.float32))
    d_gpu = th.astype(np.float64) - flat
    d_ref = th_ref.astype(np.float64) - flat
    assert np.linalg.norm(d_gpu - d_ref) / np.linalg.norm(d_ref) <= 1e-3
    # Adam from the GPU's own gradient, in the oracle: elementwise equal
    opt2 = O.Adam(flat.size, cfg)
    assert np.array_equal(opt2.step(flat, g), th)
    assert m.get_state()[3] == 1


def _gated_gpu(m, streams, pos0, n_steps, t, delta, force=()):
    import paper_2203_16114_amd as P
    ctl = P.Controller(t, delta)
    s = to_dev(streams)
    bits, ce, dec = [], [], []
    for i in range(n_steps):
        out = m.forward_bits(s, pos0 + i, 1, step_ce=True, keep=True)
        e = float(out["step_ce"][0])
        d = ctl.decide(e) | int(i in force)
        if d:
            m.adapt_step()
        bits.append(out["bits"].cpu().numpy())
        ce.append(e)
        dec.append(d)
    return np.stack(bits, 1), np.array(ce), dec


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_teacher_forced_gated_steps(dtype):
    B, n_steps, t, delta = 256, 24, 4, 0.05
    streams, _ = synth.workload_streams(4, L=2400, B=B)
    seed = 0x7ACE1004
    m = make_model(SMALL, dtype, seed, max_keep=B)
    pos0 = 2048 - 12  # straddles a source switch at 2048
    # besides the controller's own decisions, updates are forced at two steps
    # so that updates following skipped steps are covered
    force = (9, 15)
    bits, ce, dec = _gated_gpu(m, streams, pos0, n_steps, t, delta, force)
    assert t + len(force) <= sum(dec) < n_steps
    cfg = ocfg(**SMALL)
    flat = O.init_flat(cfg, seed)
    mode = "fp64" if dtype == "fp32" else "bf16"
    rbits, rce, rdec, own, _ = O.run_gated(flat, cfg, streams, pos0, n_steps, t, delta, mode=mode,
                                           forced_decisions=dec)
    tol = 1e-4 if dtype == "fp32" else 1e-3
    for s in range(n_steps):
        if dtype == "fp32":
            assert abs(ce[s] - rce[s]) <= tol, (s, ce[s], rce[s])
        else:
            assert abs(ce[s] - rce[s]) <= tol * abs(rce[s]), (s, ce[s], rce[s])
    # the host controller is bit-exact: fed the GPU's step cross-entropies, the
    # oracle's controller makes the GPU run's decisions
    c = O.Controller(t, delta)
    assert [c.decide(e) | int(s in force) for s, e in enumerate(ce)] == list(dec)
    # fed its own cross-entropies, it agrees wherever the margin to the
    # threshold is wider than the cross-entropy tolerance
    c = O.Controller(t, delta)
    for s in range(n_steps):
        thr = c.threshold() if s >= t else None
        c.decide(rce[s])
        if s not in force and (thr is None or abs(rce[s] - thr) > 2 * tol * max(1.0, abs(thr))):
            assert own[s] == dec[s], s


def test_update_is_bitwise_deterministic_and_checkpoints_resume():
    B = 512
    streams, _ = synth.workload_streams(4, L=1200, B=B)
    s = to_dev(streams)

    def run(m, p0, n):
        for i in range(n):
            m.forward_bits(s, p0 + i, 1, keep=True)
            m.adapt_step()

    a = make_model(SMALL, "bf16", 5, max_keep=B)
    b = make_model(SMALL, "bf16", 5, max_keep=B)
    run(a, 100, 5)
    run(b, 100, 3)
    th, mm, vv, step = b.get_state()
    c = make_model(SMALL, "bf16", 999, max_keep=B)
    c.set_state(th, mm, vv, step)
    run(c, 103, 2)
    sa, sc = a.get_state(), c.get_state()
    for x, y in zip(sa[:3], sc[:3]):
        assert np.array_equal(x.view(np.uint32), y.view(np.uint32))
    assert sa[3] == sc[3] == 5
    ga = a.forward_bits(s, 200, 8)["bits"]
    gc = c.forward_bits(s, 200, 8)["bits"]
    assert torch.equal(ga, gc)


def test_kept_batch_is_consumed():
    import paper_2203_16114_amd as P
    streams = synth.random_streams(2, 64, 80)
    m = make_model(SMALL, "fp32", 3, max_keep=64)
    m.forward_bits(to_dev(streams), 40, 1, keep=True)
    m.adapt_step()
    with pytest.raises(P.TraceError) as ei:
        m.adapt_step()
    assert ei.value.code == P.TRACE_ESTATE
    with pytest.raises(P.TraceError):
        m.forward_bits(to_dev(streams), 40, 2, keep=True)  # 128 windows > max_keep


def test_adapted_model_forward_matches_oracle():
    """After one update, the refreshed operand copies give the oracle's forward
    of the updated master (fp32)."""
    streams = synth.random_streams(40, 128, 120)
    m, cfg, flat, g, th, w, y = _grad_run(SMALL, "fp32", 8, streams, 60)
    out = m.forward_bits(to_dev(streams), 61, 30, logits=True)
    bb, ii = np.meshgrid(np.arange(128), 61 + np.arange(30), indexing="ij")
    w2, y2 = O.windows_at(streams, bb.ravel(), ii.ravel(), cfg.W)
    ref = O.forward(th, cfg, w2, y2, mode="fp64")
    check_parity("fp32", out["logits"].cpu().numpy(), out["bits"].cpu().numpy(), ref)
