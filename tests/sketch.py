"""Compact fingerprints of large arrays for stored expected values.

A tensor is read as rows (its first axis); each row keeps its L2 norm and its
dot products with K seeded Gaussian vectors.  Projections are linear, so the
projections of a difference are the differences of the projections, and
mean_k <e, v_k>^2 is an unbiased estimate of ||e||^2 for each row: the
difference between an array and the one a sketch came from can be measured
per row and per tensor without storing either.  Arrays of at most FULL values
are kept whole."""
from __future__ import annotations

import numpy as np

K = 4
FULL = 4096


def _rows(a):
    a = np.asarray(a, np.float64)
    return a.reshape(a.shape[0], -1) if a.ndim > 1 else a.reshape(1, -1)


def _vectors(cols: int, seed: int) -> np.ndarray:
    return np.random.default_rng(seed).standard_normal((cols, K))


def sketch(a, seed: int) -> dict:
    r = _rows(a)
    if r.size <= FULL:
        return {"shape": list(r.shape), "full": r.ravel().tolist()}
    return {"shape": list(r.shape), "norm": np.linalg.norm(r, axis=1).tolist(),
            "proj": (r @ _vectors(r.shape[1], seed)).tolist()}


def compare(sk: dict, a, seed: int):
    """(estimated ||a - ref|| / ||ref|| over the whole tensor, per-row estimated
    ||a_row - ref_row|| / ||ref_row|| as an array, per-row reference norms)."""
    r = _rows(a)
    assert list(r.shape) == sk["shape"], (r.shape, sk["shape"])
    if "full" in sk:
        ref = np.asarray(sk["full"], np.float64).reshape(r.shape)
        err = np.linalg.norm(r - ref, axis=1)
        nrm = np.linalg.norm(ref, axis=1)
    else:
        d = r @ _vectors(r.shape[1], seed) - np.asarray(sk["proj"], np.float64)
        err = np.sqrt(np.mean(d * d, axis=1))
        nrm = np.asarray(sk["norm"], np.float64)
    total = float(np.sqrt(np.sum(err ** 2)) / max(np.sqrt(np.sum(nrm ** 2)), 1e-300))
    return total, err / np.maximum(nrm, 1e-300), nrm
