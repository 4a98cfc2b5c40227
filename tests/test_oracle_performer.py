"""Pins of the oracle's Performer attention (FAVOR+, positive random features;
the backbone Sec. 6 names) against what its definition fixes: explicit loops
on tiny windows, the causal prefix-sum (linear attention) form, the estimator
of the softmax kernel of Eq. 1 as the number of features grows, and closed
forms for a zero projection and a single token."""
import math

import numpy as np
import pytest

import oracle as O
import synth

TINY = O.Config(W=8, e=4, g=2, H=2, F=12, k=1, attention="performer", n_features=6)   # T=4, d=8, dh=4


def _flat(cfg, seed, std=0.3):
    return synth.random_flat(seed, O.param_count(cfg), std)


def _phi(x, om):
    """phi(x) = m^-1/2 exp(omega x - |x|^2/2), written out (no stabiliser)."""
    m = om.shape[0]
    return np.array([math.exp(float(om[i] @ x) - 0.5 * float(x @ x)) for i in range(m)]) / math.sqrt(m)


def test_attention_weights_match_explicit_loops():
    cfg = TINY
    flat = _flat(cfg, 3)
    om = synth.performer_features(4, cfg.m, cfg.dh, orthogonal=False)
    w, y = synth.random_windows(5, 3, cfg.W)
    out = O.forward(flat, cfg, w, y, "fp64", keep=True, features=om)
    s4 = cfg.dh ** -0.25
    for n in range(3):
        for h in range(cfg.H):
            c = slice(h * cfg.dh, (h + 1) * cfg.dh)
            for t in range(cfg.T):
                pq = _phi(out["Q"][n, t, c] * s4, om)
                num = [float(pq @ _phi(out["K"][n, u, c] * s4, om)) for u in range(t + 1)]
                tot = sum(num)
                for u in range(cfg.T):
                    want = num[u] / tot if u <= t else 0.0
                    assert abs(out["A"][n, h, t, u] - want) <= 1e-12 * max(1.0, abs(want)), (n, h, t, u)


def test_causal_prefix_sum_form_equals_quadratic_form():
    """Linear attention: O_t = (sum_{u<=t} v_u phi(k_u)^T) phi(q_t) /
    (sum_{u<=t} phi(k_u))^T phi(q_t), with running sums over u."""
    cfg = O.Config(W=32, e=16, g=4, H=4, F=64, k=1, attention="performer")         # T=8, dh=16, m=128
    flat = _flat(cfg, 6, 0.2)
    om = synth.performer_features(7, cfg.m, cfg.dh)
    w, y = synth.random_windows(8, 4, cfg.W)
    out = O.forward(flat, cfg, w, y, "fp64", keep=True, features=om)
    s4 = cfg.dh ** -0.25
    for n in range(4):
        for h in range(cfg.H):
            c = slice(h * cfg.dh, (h + 1) * cfg.dh)
            S = np.zeros((cfg.m, cfg.dh))
            z = np.zeros(cfg.m)
            for t in range(cfg.T):
                fk = _phi(out["K"][n, t, c] * s4, om)
                S += np.outer(fk, out["V"][n, t, c])
                z += fk
                fq = _phi(out["Q"][n, t, c] * s4, om)
                o = (fq @ S) / (fq @ z)
                np.testing.assert_allclose(out["O"][n, t, c], o, rtol=1e-10, atol=1e-13)


def test_features_estimate_the_softmax_kernel():
    """E over omega ~ N(0, I) of phi(q')^T phi(k') is exp(q'.k') = exp(q.k /
    sqrt(dh)), the kernel of Eq. 1: with many features the estimate matches
    it within its Monte Carlo error, and the attention weights approach the
    softmax weights."""
    dh, m = 16, 1 << 17
    r = np.random.default_rng(11)
    om = synth.performer_features(12, m, dh, orthogonal=False).astype(np.float64)
    for _ in range(5):
        q, k = r.standard_normal(dh) * 0.5, r.standard_normal(dh) * 0.5
        s4 = dh ** -0.25
        terms = np.exp(om @ (q * s4) - 0.5 * (q * s4) @ (q * s4)) * np.exp(om @ (k * s4) - 0.5 * (k * s4) @ (k * s4))
        est, se = terms.mean(), terms.std() / math.sqrt(m)
        assert abs(est - math.exp(q @ k / math.sqrt(dh))) < 5 * se
    Qh = r.standard_normal((3, 8, dh)) * 0.5
    Kh = r.standard_normal((3, 8, dh)) * 0.5
    A = O.performer_attention_weights(Qh, Kh, om, np.float64)
    S = np.einsum("ntc,nuc->ntu", Qh, Kh) / math.sqrt(dh)
    S = np.where(np.tril(np.ones((8, 8), bool))[None], S, -np.inf)
    np.testing.assert_allclose(A, O.softmax_lastaxis(S), rtol=0, atol=1e-2)


def test_zero_projection_and_single_token_closed_forms():
    dh = 8
    r = np.random.default_rng(13)
    Qh = r.standard_normal((2, 4, dh))
    Kh = r.standard_normal((2, 4, dh))
    A = O.performer_attention_weights(Qh, Kh, np.zeros((32, dh)), np.float64)
    # omega = 0: phi(x) = m^-1/2 exp(-|x|^2/2) 1, so A[t, u] is prop. to exp(-|k'_u|^2 / 2)
    g = np.exp(-0.5 * np.sum((Kh * dh ** -0.25) ** 2, axis=-1))
    for t in range(4):
        want = g[:, :t + 1] / g[:, :t + 1].sum(1, keepdims=True)
        np.testing.assert_allclose(A[:, t, :t + 1], want, rtol=1e-13)
        assert np.all(A[:, t, t + 1:] == 0)
    A1 = O.performer_attention_weights(Qh[:, :1], Kh[:, :1], r.standard_normal((32, dh)), np.float64)
    assert np.all(A1 == 1.0)


def test_orthogonal_features_are_orthogonal_blocks_with_gaussian_norms():
    dh, m = 32, 128
    om = synth.performer_features(21, m, dh).astype(np.float64)
    assert om.shape == (m, dh)
    for b in range(m // dh):
        blk = om[b * dh:(b + 1) * dh]
        G = blk @ blk.T
        np.testing.assert_allclose(G - np.diag(np.diag(G)), 0, atol=1e-4 * np.max(np.diag(G)))
    n2 = np.sum(om ** 2, axis=1)
    assert abs(n2.mean() - dh) < 4 * math.sqrt(2 * dh / m)       # chi-square(dh) norms


def test_bf16_mode_rounds_the_projection_like_a_weight():
    cfg = O.Config(W=16, e=16, g=4, H=2, F=64, k=1, attention="performer")
    flat = O.init_flat(cfg, 1, 0.1)
    om = synth.performer_features(2, cfg.m, cfg.dh)
    w, y = synth.random_windows(3, 8, cfg.W)
    a = O.forward(flat, cfg, w, y, "bf16", features=om)["z"]
    b = O.forward(flat, cfg, w, y, "bf16", features=O.bf16_round(om))["z"]
    assert np.array_equal(a, b)
    with pytest.raises(ValueError):
        O.forward(flat, cfg, w, y, "bf16")
