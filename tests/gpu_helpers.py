"""Helpers for the GPU parity tests: models built through the C ABI from a
workload's shape, seeded inputs, and the comparison rules."""
from __future__ import annotations

import numpy as np

import oracle as O
from synth import WORKLOADS


def ocfg(W, e, g, H, F, k, use_pos=True):
    return O.Config(W=W, e=e, g=g, H=H, F=F, k=k, use_pos=use_pos)


def workload_cfg(wid):
    w = WORKLOADS[wid]
    return dict(W=w.W, e=w.e, g=w.g, H=w.H, F=w.F, k=w.k), w.dtype


def make_model(shape, dtype, seed, max_windows=1 << 16, max_keep=0, use_pos=True, flat=None):
    import paper_2203_16114_amd as P
    m = P.TraceModel(**shape, dtype=dtype, use_pos=use_pos, max_windows=max_windows, max_keep=max_keep)
    m.init_weights(seed, 0.02, flat)
    return m


def to_dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def row_rel_err(z, zref):
    """Per-row relative logit error ||z - zref||_inf / max(||zref||_inf, 1e-6)."""
    z = np.asarray(z, np.float64)
    zref = np.asarray(zref, np.float64)
    num = np.max(np.abs(z - zref), axis=1)
    den = np.maximum(np.max(np.abs(zref), axis=1), 1e-6)
    return num / den


def oracle_mode(dtype):
    return "fp64" if dtype == "fp32" else "bf16"


def check_parity(dtype, z, bits, ref):
    """The tolerances of the forward parity bar: fp32 (oracle in fp64) logits
    rel 1e-4 per row and bits/byte abs 1e-4; bf16 (oracle emulating the bf16
    storage points) logits rel 2e-2 and bits/byte rel 1e-3."""
    rel = row_rel_err(z, ref["z"])
    bpb = float(np.mean(np.asarray(bits, np.float64)))
    bpb_ref = float(np.mean(np.asarray(ref["bits"], np.float64)))
    if dtype == "fp32":
        assert rel.max() <= 1e-4, f"logit rel err {rel.max():.3e}"
        assert abs(bpb - bpb_ref) <= 1e-4, f"bits/byte {bpb} vs {bpb_ref}"
    else:
        assert rel.max() <= 2e-2, f"logit rel err {rel.max():.3e}"
        assert abs(bpb - bpb_ref) <= 1e-3 * abs(bpb_ref), f"bits/byte {bpb} vs {bpb_ref}"
    return rel.max(), abs(bpb - bpb_ref)


def structured_flat(cfg, sel):
    """Weights under which every logit is one byte-embedding value of one slot
    of one token, so that the logits show, exactly, which byte each kernel put
    in each slot (Sec. 4.2).

    E[v][c] = (v + 37 c) mod 256 for c in a set S of components (a bijection of
    v for each c; other components 0); position t is a one-hot P[t] in a
    component E leaves at zero.  K_h of token u is the one-hot of u and q_h
    scores -1024 on every token but sel[h], so head h attends to token sel[h]
    alone (weight exactly 1); V_h copies that token's S components of every
    slot; Wo moves them to dimensions where the last token's own X is zero;
    W1 = W2 = 0 (the FFN adds exactly 0); Wout copies the last token's S
    components and the heads' outputs to the first logits.  Every value is an
    integer below 256 (exact in bf16) or a one-hot weight.
    Returns (flat, expected logits as a function of the windows)."""
    T, g, e, d, H, dh = cfg.T, cfg.g, cfg.e, cfg.d, cfg.H, cfg.dh
    npos = -(-T // g)
    s = min((e - npos) // (H + 1), 256 // (g * (H + 1)), dh // g)
    S = [0] + list(range(1 + npos, npos + s))
    assert len(S) == s >= 1
    p = {n: np.zeros(shape, np.float32) for n, shape in O.param_layout(cfg)}
    v = np.arange(256)
    for c in S:
        p["E"][:, c] = (v + 37 * c) % 256
    prow = lambda t: (t % g) * e + 1 + t // g          # the component of position t
    for t in range(T):
        p["P"][t, prow(t)] = 1.0
    for h in range(H):
        for u in range(T):
            p["Wk"][prow(u), h * dh + u] = 1.0
            p["Wq"][prow(T - 1), h * dh + u] = 0.0 if u == sel[h] else -1024.0
        for x in range(g):
            for ci, c in enumerate(S):
                p["Wv"][x * e + c, h * dh + x * s + ci] = 1.0
    free = [x * e + c for x in range(g) for c in range(e) if c not in S and not (1 <= c <= npos)]
    assert H * g * s <= len(free)
    k = 0
    for h in range(H):
        for j in range(g * s):
            p["Wo"][h * dh + j, free[k]] = 1.0
            k += 1
    last = [x * e + c for x in range(g) for c in S]
    for i, dim in enumerate(last + free[:H * g * s]):
        p["Wout"][dim, i] = 1.0
    flat = O.flatten(p, cfg, np.float32)

    def expected(win):
        N = win.shape[0]
        z = np.zeros((N, 256), np.float32)
        for x in range(g):
            for ci, c in enumerate(S):
                z[:, x * s + ci] = (win[:, (T - 1) * g + x].astype(np.int64) + 37 * c) % 256
        base = g * s
        for h in range(H):
            for x in range(g):
                for ci, c in enumerate(S):
                    z[:, base + h * g * s + x * s + ci] = (win[:, sel[h] * g + x].astype(np.int64) + 37 * c) % 256
        return z
    return flat, expected
