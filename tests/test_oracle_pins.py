"""Pins of the CPU oracle against what the paper and the mathematics fix.

None of these re-types the oracle's own formula: each checks it against brute
force on tiny inputs, a closed form, an invariant, a library routine or a
hand-evaluated example (tests/golden/)."""
import json
import math
import os

import numpy as np
import pytest
import scipy.stats
import torch

import oracle as O
import synth

HERE = os.path.dirname(os.path.abspath(__file__))

TINY = O.Config(W=8, e=4, g=2, H=2, F=12, k=2)          # T=4, d=8, dh=4
C1 = O.Config(W=16, e=16, g=4, H=1, F=256, k=2)


def _flat(cfg, seed, std=0.3):
    return synth.random_flat(seed, O.param_count(cfg), std)


# ------------------------------------------------------------------ rounding
def test_bf16_round_matches_torch_rne():
    r = np.random.default_rng(0)
    x = np.concatenate([r.standard_normal(100000).astype(np.float32) * 10 ** r.uniform(-30, 30, 100000).astype(np.float32),
                        np.array([0.0, -0.0, 1.0, 1.00390625, 1.01171875, 3.4e38, -3.4e38, 1e-40, np.inf, -np.inf],
                                 np.float32)])
    want = torch.from_numpy(x).to(torch.bfloat16).float().numpy()
    got = O.bf16_round(x)
    assert np.array_equal(got.view(np.uint32), want.view(np.uint32))
    assert np.isnan(O.bf16_round(np.array([np.nan], np.float32)))[0]


# ------------------------------------------------------------------ windows
def test_windows_are_the_previous_W_bytes_oldest_first():
    s = synth.random_streams(1, 3, 50)
    w, y = O.windows_at(s, np.array([0, 2, 1]), np.array([8, 49, 20]), 8)
    assert np.array_equal(w[0], s[0, 0:8]) and y[0] == s[0, 8]
    assert np.array_equal(w[1], s[2, 41:49]) and y[1] == s[2, 49]
    assert np.array_equal(w[2], s[1, 12:20]) and y[2] == s[1, 20]
    with pytest.raises(ValueError):
        O.windows_at(s, np.array([0]), np.array([7]), 8)
    wa, ya = O.all_windows(s, 8)
    assert wa.shape == (3 * 42, 8)
    assert np.array_equal(wa[42 + 5], s[1, 5:13]) and ya[42 + 5] == s[1, 13]


# ------------------------------------------------------------------ grouping
@pytest.mark.parametrize("cfg", [TINY, C1, O.Config(W=6, e=5, g=1, H=1, F=4, k=1)])
def test_group_gather_matches_index_formula(cfg):
    flat = _flat(cfg, 3)
    p = O.compute_params(flat, cfg, "fp64")
    w, _ = synth.random_windows(4, 9, cfg.W)
    X = O.embed_group(p, w, cfg, O.trace_oracle._Mode("fp64"))
    r = np.random.default_rng(5)
    for _ in range(300):
        n, t, j, c = r.integers(9), r.integers(cfg.T), r.integers(cfg.g), r.integers(cfg.e)
        want = p["E"][w[n, t * cfg.g + j], c] + p["P"][t, j * cfg.e + c]
        assert X[n, t, j * cfg.e + c] == want
    if cfg.g == 1:   # g = 1 is a plain per-byte embedding
        assert np.array_equal(X, p["E"][w] + p["P"][None])


# ----------------------------------------------------------------- attention
def _brute_attention_layer0(flat, cfg, w):
    """Eqs. 1-2 and the inner residual of Eq. 4 with explicit loops (fp64)."""
    p = O.unflatten(np.asarray(flat, np.float64), cfg)
    N, T, d, H, dh = w.shape[0], cfg.T, cfg.d, cfg.H, cfg.dh
    Y0 = np.zeros((N, T, d))
    for n in range(N):
        X = np.zeros((T, d))
        for t in range(T):
            for b in range(cfg.g):
                for c in range(cfg.e):
                    X[t, b * cfg.e + c] = p["E"][w[n, t * cfg.g + b], c] + p["P"][t, b * cfg.e + c]
        Q = np.zeros((T, d)); K = np.zeros((T, d)); V = np.zeros((T, d))
        for t in range(T):
            for o in range(d):
                Q[t, o] = sum(X[t, c] * p["Wq"][c, o] for c in range(d))
                K[t, o] = sum(X[t, c] * p["Wk"][c, o] for c in range(d))
                V[t, o] = sum(X[t, c] * p["Wv"][c, o] for c in range(d))
        heads = np.zeros((T, d))
        for h in range(H):
            for t in range(T):
                sc = [sum(Q[t, h * dh + c] * K[u, h * dh + c] for c in range(dh)) / math.sqrt(dh)
                      for u in range(t + 1)]
                mx = max(sc)
                ex = [math.exp(s - mx) for s in sc]
                tot = sum(ex)
                for c in range(dh):
                    heads[t, h * dh + c] = sum(ex[u] / tot * V[u, h * dh + c] for u in range(t + 1))
        for t in range(T):
            for o in range(d):
                Y0[n, t, o] = sum(heads[t, c] * p["Wo"][c, o] for c in range(d)) + X[t, o]
    return Y0


@pytest.mark.parametrize("cfg", [TINY, O.Config(W=6, e=3, g=2, H=1, F=5, k=1)])
def test_attention_matches_brute_force(cfg):
    flat = _flat(cfg, 7)
    w, y = synth.random_windows(8, 4, cfg.W)
    out = O.forward(flat, cfg, w, y, "fp64", keep=True)
    np.testing.assert_allclose(out["Y"][0], _brute_attention_layer0(flat, cfg, w), rtol=1e-12, atol=1e-14)


def test_single_token_attention_is_value_then_output_projection():
    cfg = O.Config(W=4, e=2, g=4, H=2, F=6, k=1)     # T = 1: softmax of one score is 1
    flat = _flat(cfg, 9)
    p = O.unflatten(np.asarray(flat, np.float64), cfg)
    w, y = synth.random_windows(10, 5, cfg.W)
    out = O.forward(flat, cfg, w, y, "fp64", keep=True)
    X = out["X"][:, 0, :]
    np.testing.assert_allclose(out["Y"][0][:, 0, :] - X, X @ p["Wv"] @ p["Wo"], rtol=1e-12, atol=1e-15)


def test_zero_query_gives_uniform_mean_of_values():
    cfg = TINY
    flat = _flat(cfg, 11).astype(np.float64)
    p = O.unflatten(flat, cfg)
    p["Wq"][:] = 0
    w, y = synth.random_windows(12, 5, cfg.W)
    out = O.forward(flat, cfg, w, y, "fp64", keep=True)
    V = out["X"] @ p["Wv"]
    for t in range(cfg.T):
        np.testing.assert_allclose(out["O"][:, t, :], V[:, :t + 1, :].mean(axis=1), rtol=1e-12, atol=1e-15)


def test_attention_is_causal():
    cfg = TINY
    flat = _flat(cfg, 13)
    w, y = synth.random_windows(14, 6, cfg.W)
    base = O.forward(flat, cfg, w, y, "fp64", keep=True)
    for t in range(cfg.T - 1):
        w2 = w.copy()
        w2[:, (t + 1) * cfg.g:] = ((w2[:, (t + 1) * cfg.g:].astype(np.int64) + 77) % 256).astype(np.uint8)   # perturb tokens u > t
        o2 = O.forward(flat, cfg, w2, y, "fp64", keep=True)
        np.testing.assert_array_equal(o2["Y"][cfg.k][:, :t + 1], base["Y"][cfg.k][:, :t + 1])
        assert not np.allclose(o2["Y"][cfg.k][:, t + 1:], base["Y"][cfg.k][:, t + 1:])


# ----------------------------------------------------------------------- FFN
def test_gelu_is_x_times_normal_cdf():
    u = np.linspace(-7, 7, 1001)
    np.testing.assert_allclose(O.gelu(u), u * scipy.stats.norm.cdf(u), rtol=1e-13, atol=1e-300)
    assert O.gelu(np.zeros(1))[0] == 0.0


def test_ffn_with_zero_W2_is_identity():
    cfg = TINY
    flat = _flat(cfg, 15).astype(np.float64)
    O.unflatten(flat, cfg)["W2"][:] = 0
    w, y = synth.random_windows(16, 4, cfg.W)
    out = O.forward(flat, cfg, w, y, "fp64", keep=True)
    for r in range(1, cfg.k + 1):
        np.testing.assert_array_equal(out["Y"][r], out["Y"][0])


def test_k1_layer_is_eq4_literally_and_k2_composes_the_same_ffn():
    cfg1 = O.Config(W=8, e=4, g=2, H=2, F=12, k=1)
    cfg2 = O.Config(W=8, e=4, g=2, H=2, F=12, k=2)
    flat = _flat(cfg1, 17).astype(np.float64)
    p = O.unflatten(flat, cfg1)
    w, y = synth.random_windows(18, 4, cfg1.W)
    o1 = O.forward(flat, cfg1, w, y, "fp64", keep=True)
    att_plus_x = o1["Y"][0]                                 # Attention(x) + x
    ffn = lambda v: (v @ p["W1"]) * scipy.stats.norm.cdf(v @ p["W1"]) @ p["W2"]   # noqa: E731
    np.testing.assert_allclose(o1["Y"][1], ffn(att_plus_x) + att_plus_x, rtol=1e-12, atol=1e-15)
    o2 = O.forward(flat, cfg2, w, y, "fp64", keep=True)
    y1 = ffn(att_plus_x) + att_plus_x
    np.testing.assert_allclose(o2["Y"][2], ffn(y1) + y1, rtol=1e-12, atol=1e-15)


# ---------------------------------------------------------------------- head
@pytest.mark.parametrize("mode", ["fp64", "fp32", "bf16"])
def test_zeroed_head_gives_exactly_8_bits(mode):
    cfg = C1
    flat = _flat(cfg, 19, 0.02)
    p = O.unflatten(flat, cfg)
    p["Wout"][:] = 0
    p["bout"][:] = 0
    w, y = synth.random_windows(20, 64, cfg.W)
    out = O.forward(flat, cfg, w, y, mode)
    assert np.all(out["bits"] == 8.0)


def test_bias_only_head_gives_minus_log2_q():
    cfg = C1
    flat = _flat(cfg, 21, 0.02).astype(np.float64)
    p = O.unflatten(flat, cfg)
    q = np.random.default_rng(22).dirichlet(np.ones(256) * 0.5)
    q = np.maximum(q, 1e-12); q /= q.sum()
    p["Wout"][:] = 0
    p["bout"][:] = np.log(q)
    w, y = synth.random_windows(23, 200, cfg.W)
    out = O.forward(flat, cfg, w, y, "fp64")
    np.testing.assert_allclose(out["bits"], -np.log2(q[y]), rtol=1e-12)


def test_bias_only_head_on_iid_zipf_reaches_source_entropy():
    cfg = C1
    cdf = synth.zipf_table(1.2, 99)
    q = synth.cdf_probs(cdf)
    streams, codelen = synth.generate([(synth.SRC_ZIPF, 0, cdf)], np.zeros((4, 1), np.int32), 4096, 4096,
                                      np.arange(1, 5, dtype=np.uint64))
    flat = _flat(cfg, 24, 0.02).astype(np.float64)
    p = O.unflatten(flat, cfg)
    p["Wout"][:] = 0
    p["bout"][:] = np.log(np.maximum(q, 1e-300))
    w, y = O.all_windows(streams, cfg.W)
    bits = O.forward(flat, cfg, w, y, "fp64")["bits"]
    H = -(q * np.log2(np.maximum(q, 1e-300))).sum()
    assert abs(H - 5.2898) < 1e-3                        # Zipf(1.2) over 256 symbols
    assert abs(O.bits_per_byte(bits) - H) < 0.05         # empirical cross-entropy ~ H
    # the generator's own code length of the same bytes agrees with -log2 q
    np.testing.assert_allclose(bits.reshape(4, -1).sum(1),
                               codelen - np.array([-np.log2(q[s]).sum() for s in streams[:, :cfg.W]]),
                               rtol=1e-9)


@pytest.mark.parametrize("mode", ["fp64", "fp32"])
def test_softmax_rows_sum_to_one_and_bits_are_minus_log2_p(mode):
    cfg = C1
    flat = _flat(cfg, 25, 0.06)
    w, y = synth.random_windows(26, 300, cfg.W)
    out = O.forward(flat, cfg, w, y, mode)
    z = np.asarray(out["z"], np.float64)
    P = np.exp(z - z.max(1, keepdims=True)); P /= P.sum(1, keepdims=True)
    Pm = O.softmax_lastaxis(out["z"])
    assert np.max(np.abs(Pm.sum(1) - 1)) < (1e-6 if mode == "fp32" else 1e-14)
    tol = 2e-5 if mode == "fp32" else 1e-12
    np.testing.assert_allclose(out["bits"], -np.log2(P[np.arange(300), y]), rtol=tol, atol=tol)
    # bits/byte is the mean of -log2 p
    assert abs(O.bits_per_byte(out["bits"]) - float(np.mean(-np.log2(P[np.arange(300), y])))) < tol


def test_stream_bits_per_byte_charges_first_W_bytes_8_bits():
    assert O.stream_bits_per_byte(0.0, 2, 10, 4) == pytest.approx(8 * 4 * 2 / 20)
    assert O.stream_bits_per_byte(8.0 * 12, 2, 10, 4) == pytest.approx(8.0)


# --------------------------------------------------------------------- lanes
def test_permuting_batch_lanes_permutes_outputs():
    cfg = TINY
    flat = _flat(cfg, 27)
    w, y = synth.random_windows(28, 33, cfg.W)
    perm = np.random.default_rng(29).permutation(33)
    a = O.forward(flat, cfg, w, y, "fp64")
    b = O.forward(flat, cfg, w[perm], y[perm], "fp64")
    np.testing.assert_allclose(b["z"], a["z"][perm], rtol=1e-13, atol=1e-15)
    _, ga = O.forward_backward(flat, cfg, w, y)
    _, gb = O.forward_backward(flat, cfg, w[perm], y[perm])
    for n in ga:
        np.testing.assert_allclose(gb[n], ga[n], rtol=1e-10, atol=1e-15)


# ------------------------------------------------------------------ backward
@pytest.mark.parametrize("cfg", [TINY, O.Config(W=8, e=4, g=2, H=2, F=12, k=3, use_pos=False),
                                 O.Config(W=4, e=3, g=1, H=3, F=7, k=1)])
def test_gradients_match_central_finite_differences(cfg):
    flat = _flat(cfg, 31, 0.4).astype(np.float64)
    w, y = synth.random_windows(32, 6, cfg.W)
    w[0, :2] = w[1, 2:4]                     # repeated bytes: E rows receive several scatters
    _, g = O.forward_backward(flat, cfg, w, y, "fp64")
    gflat = O.flatten(g, cfg)
    r = np.random.default_rng(33)
    off = 0
    worst = 0.0
    for name, shape in O.param_layout(cfg):
        n = int(np.prod(shape))
        if name == "E":   # rows of bytes that occur, so the gradient is non-trivial
            rows = np.unique(w)
            idx = [int(rows[r.integers(len(rows))]) * cfg.e + int(r.integers(cfg.e)) for _ in range(6)]
        else:
            idx = r.choice(n, size=min(6, n), replace=False)
        for i in idx:
            j = off + int(i)
            h = 1e-6 * max(1.0, abs(flat[j]))
            fp = flat.copy(); fp[j] += h
            fm = flat.copy(); fm[j] -= h
            fd = (O.loss_nats(fp, cfg, w, y) - O.loss_nats(fm, cfg, w, y)) / (2 * h)
            err = abs(fd - gflat[j])
            assert err <= 1e-6 * abs(gflat[j]) + 2e-9, (name, i, fd, gflat[j])
            worst = max(worst, err)
        off += n
    if not cfg.use_pos:
        assert np.all(g["P"] == 0)


# ---------------------------------------------------------------------- Adam
def test_first_adam_step_is_minus_lr_sign_like():
    cfg = TINY
    n = O.param_count(cfg)
    r = np.random.default_rng(35)
    theta = r.standard_normal(n).astype(np.float32)
    g = (r.standard_normal(n) * 10.0 ** r.uniform(-6, 1, n)).astype(np.float32)
    opt = O.Adam(n, cfg)
    new = opt.step(theta, g)
    want = -1e-3 * g.astype(np.float64) / (np.abs(g.astype(np.float64)) + 1e-8)
    np.testing.assert_allclose(new.astype(np.float64) - theta, want, rtol=2e-3, atol=2e-7)
    assert opt.tau == 1
    # second step against the recurrence written out in float64
    g2 = (r.standard_normal(n) * 1e-3).astype(np.float32)
    new2 = opt.step(new, g2)
    g1d, g2d = g.astype(np.float64), g2.astype(np.float64)
    m = 0.9 * (0.1 * g1d) + 0.1 * g2d
    v = 0.999 * (0.001 * g1d * g1d) + 0.001 * g2d * g2d
    step = 1e-3 * (m / (1 - 0.9 ** 2)) / (np.sqrt(v / (1 - 0.999 ** 2)) + 1e-8)
    np.testing.assert_allclose(new2.astype(np.float64), new.astype(np.float64) - step, rtol=0, atol=3e-7)
    assert opt.tau == 2


# ---------------------------------------------------------------- controller
def test_controller_worked_example():
    ex = json.load(open(os.path.join(HERE, "golden", "controller_worked_example.json")))
    c = O.Controller(ex["t"], ex["delta"])
    thr, dec = [], []
    for i, e in enumerate(ex["ce"]):
        if i >= ex["t"]:
            thr.append(c.threshold())
        dec.append(c.decide(e))
    assert dec == ex["decisions"]
    np.testing.assert_allclose(thr, ex["thresholds_from_step_4"], rtol=0, atol=1e-12)
    assert 5.75 + 0.05 == 5.8    # the tie really is a tie in IEEE double


def test_controller_is_o1_fifo_of_last_t():
    r = np.random.default_rng(36)
    for t in (1, 3, 16, 256):
        c = O.Controller(t, 0.0)
        seq = r.uniform(0, 8, 2000)
        for i, e in enumerate(seq):
            d = c.decide(e)
            if i >= t:
                mean = float(np.mean(seq[i - t:i]))
                if abs(e - mean) > 1e-9:
                    assert d == int(e > mean)
            else:
                assert d == 1
        assert c.ring == list(seq[-t:])
    with pytest.raises(ValueError):
        O.Controller(0, 0.0)
    with pytest.raises(ValueError):
        O.Controller(4, 0.0).decide(float("nan"))


# -------------------------------------------------------------------- init
def test_init_is_seeded_normal_with_zero_bias():
    cfg = O.Config(W=32, e=32, g=4, H=4, F=512, k=2)
    a = O.init_flat(cfg, 1234)
    b = O.init_flat(cfg, 1234)
    c = O.init_flat(cfg, 1235)
    assert np.array_equal(a, b) and not np.array_equal(a, c)
    p = O.unflatten(a, cfg)
    assert np.all(p["bout"] == 0)
    body = a[:-256].astype(np.float64)
    assert abs(body.mean()) < 3 * 0.02 / math.sqrt(body.size) * 2
    assert abs(body.std() - 0.02) < 2e-4
    assert scipy.stats.kstest(body / 0.02, "norm").pvalue > 1e-3
    assert O.param_count(cfg) == 238848


def test_untied_ffn_with_equal_copies_is_the_shared_ffn():
    """Sec. 6.3's untied FFN with every repeat's W1, W2 equal to the shared
    ones computes the shared FFN of Sec. 4.3; its per-repeat gradients sum to
    the shared gradient."""
    tied = O.Config(W=16, e=16, g=4, H=2, F=64, k=3)
    unt = O.Config(W=16, e=16, g=4, H=2, F=64, k=3, untied=True)
    ft = O.init_flat(tied, 5)
    pt = O.unflatten(ft, tied)
    pu = dict(pt)
    pu["W1"] = np.stack([pt["W1"]] * 3)
    pu["W2"] = np.stack([pt["W2"]] * 3)
    fu = O.flatten(pu, unt, np.float64)
    assert fu.size == O.param_count(tied) + 2 * 2 * 64 * 64      # two more copies of W1 and W2 (d = 64)
    rng = np.random.default_rng(2)
    streams = rng.integers(0, 256, (3, 40)).astype(np.uint8)
    w, y = O.windows_at(streams, np.array([0, 1, 2, 0]), np.array([16, 20, 39, 30]), 16)
    rt, gt = O.forward_backward(ft, tied, w, y)
    ru, gu = O.forward_backward(fu, unt, w, y)
    assert np.allclose(rt["bits"], ru["bits"], rtol=0, atol=1e-12)
    assert np.allclose(gu["W1"].sum(0), gt["W1"], atol=1e-12) and np.allclose(gu["W2"].sum(0), gt["W2"], atol=1e-12)
    assert np.allclose(gu["Wq"], gt["Wq"], atol=1e-12)
    # different copies: the repeats are no longer interchangeable
    pu["W1"][1] *= 1.5
    r2 = O.forward(O.flatten(pu, unt, np.float64), unt, w, y)
    assert np.max(np.abs(r2["bits"] - ru["bits"])) > 1e-7


# ------------------------------------------ structured weights (index test)
@pytest.mark.parametrize("shape", [dict(W=16, e=16, g=4, H=1, F=256, k=2), dict(W=32, e=32, g=4, H=4, F=512, k=2),
                                   dict(W=64, e=32, g=8, H=8, F=1024, k=3), dict(W=64, e=64, g=8, H=8, F=2048, k=3)])
def test_structured_weights_show_every_slot_exactly(shape):
    """The weights of the GPU index test make the oracle's logits (fp64 and
    bf16 emulation) equal, exactly, the byte-embedding values the index map of
    Sec. 4.2 puts in each slot of the selected tokens; a window with two slots
    of one token exchanged gives different logits."""
    from gpu_helpers import structured_flat
    cfg = O.Config(**shape)
    w, y = synth.random_windows(61, 40, cfg.W)
    for r in range(-(-cfg.T // cfg.H)):
        sel = [(r * cfg.H + h) % cfg.T for h in range(cfg.H)]
        flat, expected = structured_flat(cfg, sel)
        want = expected(w)
        for mode in ("fp64", "bf16"):
            z = np.asarray(O.forward(flat, cfg, w, y, mode)["z"], np.float32)
            assert np.array_equal(z.view(np.uint32), want.view(np.uint32)), mode
        t = sel[0]
        sw = w.copy()
        sw[:, [t * cfg.g, t * cfg.g + 1]] = sw[:, [t * cfg.g + 1, t * cfg.g]]
        diff = np.any(expected(sw) != want, axis=1)
        assert np.array_equal(diff, w[:, t * cfg.g] != w[:, t * cfg.g + 1])


# ---------------------------------------------------------------- layers > 1
@pytest.mark.parametrize("cfg", [O.Config(W=8, e=4, g=2, H=2, F=12, k=2, layers=2),
                                 O.Config(W=8, e=4, g=2, H=2, F=12, k=2, layers=3, use_pos=False),
                                 O.Config(W=8, e=4, g=2, H=2, F=12, k=2, layers=2, untied=True)])
def test_multilayer_gradients_match_central_finite_differences(cfg):
    flat = _flat(cfg, 41, 0.4).astype(np.float64)
    w, y = synth.random_windows(42, 5, cfg.W)
    _, g = O.forward_backward(flat, cfg, w, y, "fp64")
    gflat = O.flatten(g, cfg)
    # central differences carry a round-off of about 1e-16 |loss| / h
    floor = 2e-9 * max(1.0, O.loss_nats(flat, cfg, w, y))
    r = np.random.default_rng(43)
    off = 0
    for name, shape in O.param_layout(cfg):
        n = int(np.prod(shape))
        if name == "E":
            rows = np.unique(w)
            idx = [int(rows[r.integers(len(rows))]) * cfg.e + int(r.integers(cfg.e)) for _ in range(6)]
        else:
            idx = r.choice(n, size=min(8, n), replace=False)
        for i in idx:
            j = off + int(i)
            h = 1e-6 * max(1.0, abs(flat[j]))
            fp = flat.copy(); fp[j] += h
            fm = flat.copy(); fm[j] -= h
            fd = (O.loss_nats(fp, cfg, w, y) - O.loss_nats(fm, cfg, w, y)) / (2 * h)
            assert abs(fd - gflat[j]) <= 1e-6 * abs(gflat[j]) + floor, (name, i, fd, gflat[j])
        off += n


def test_pass_through_layer_and_layer_count():
    """A layer with Wv = Wo = W2 = 0 adds exactly zero to its input (Eq. 4's
    two residuals carry it through), so a 2-layer model whose first layer is
    one computes the 1-layer model with the second layer's weights; the
    parameter count grows by one set of Wq .. W2 per layer."""
    one = O.Config(W=16, e=8, g=4, H=2, F=32, k=2)
    two = O.Config(W=16, e=8, g=4, H=2, F=32, k=2, layers=2)
    f1 = _flat(one, 44, 0.2).astype(np.float64)
    p1 = O.unflatten(f1, one)
    p2 = {n: np.array(v) for n, v in p1.items()}
    rng = np.random.default_rng(45)
    for n in ("Wq", "Wk", "Wv", "Wo", "W1", "W2"):
        first = rng.standard_normal(p1[n].shape) * 0.2
        if n in ("Wv", "Wo", "W2"):
            first[:] = 0
        p2[n] = np.stack([first, p1[n]])
    f2 = O.flatten(p2, two, np.float64)
    assert f2.size == O.param_count(one) + 4 * 32 * 32 + 2 * 32 * 32
    w, y = synth.random_windows(46, 7, 16)
    a = O.forward(f1, one, w, y, "fp64")
    b = O.forward(f2, two, w, y, "fp64", keep=True)
    np.testing.assert_allclose(b["z"], a["z"], rtol=1e-12, atol=1e-12)
    np.testing.assert_array_equal(b["layers"][0]["Y"][-1], b["layers"][0]["X"])


def test_multilayer_rows_are_causal():
    """Row t of every layer's output depends only on tokens u <= t."""
    cfg = O.Config(W=16, e=8, g=4, H=2, F=32, k=1, layers=3)
    flat = _flat(cfg, 47, 0.3).astype(np.float64)
    w, y = synth.random_windows(48, 4, 16)
    a = O.forward(flat, cfg, w, y, "fp64", keep=True)
    for t in range(cfg.T - 1):
        w2 = w.copy()
        w2[:, (t + 1) * cfg.g:] ^= 0x33               # every token after t changes
        b = O.forward(flat, cfg, w2, y, "fp64", keep=True)
        for l in range(cfg.layers):
            np.testing.assert_array_equal(b["layers"][l]["Y"][-1][:, :t + 1], a["layers"][l]["Y"][-1][:, :t + 1])
        assert not np.allclose(b["layers"][-1]["Y"][-1][:, t + 1:], a["layers"][-1]["Y"][-1][:, t + 1:])
