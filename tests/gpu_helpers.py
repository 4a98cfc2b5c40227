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
