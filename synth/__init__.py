"""Seeded synthetic inputs shared by the oracle tests, the GPU tests and the
benchmark.  Holds workload shapes and byte-stream sources only; none of the
estimator's arithmetic lives here.

The paper's datasets (Enwik8/9, BookCorpus, ESC audio, ImageNet, Spitzer float
data, a disk backup, Silesia; Sec. 6 and App. A Table 5) are not available; the
sources below stand in for their mix of homogeneous and heterogeneous byte
streams: order-k Markov sources with Dirichlet rows, Zipf byte distributions
over a seeded permutation, uniform bytes and geometric runs of repeated bytes.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

from .workloads import WORKLOADS, Workload  # noqa: F401

_HERE = os.path.dirname(os.path.abspath(__file__))
_SO = os.path.join(_HERE, "_gen.so")
_lib = None

SRC_MARKOV, SRC_ZIPF, SRC_UNIFORM, SRC_RUNS = 0, 1, 2, 3


class _Source(ctypes.Structure):
    _fields_ = [("type", ctypes.c_int32), ("order", ctypes.c_int32), ("cdf", ctypes.c_void_p)]


def build(force: bool = False) -> str:
    """Compile gen.c into _gen.so with gcc (OpenMP, no fast-math)."""
    if force or not os.path.exists(_SO):
        tmp = _SO + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-shared", "-fPIC", "-o", tmp,
                               os.path.join(_HERE, "gen.c"), "-lm"])
        os.replace(tmp, _SO)
    return _SO


def lib():
    global _lib
    if _lib is None:
        build()
        L = ctypes.CDLL(_SO)
        L.synth_splitmix64.restype = ctypes.c_uint64
        L.synth_splitmix64.argtypes = [ctypes.c_uint64]
        L.synth_markov_rows.restype = ctypes.c_int64
        L.synth_markov_rows.argtypes = [ctypes.c_int]
        L.synth_markov_table.restype = ctypes.c_int
        L.synth_markov_table.argtypes = [ctypes.c_int, ctypes.c_double, ctypes.c_uint64, ctypes.c_void_p]
        L.synth_zipf_table.restype = ctypes.c_int
        L.synth_zipf_table.argtypes = [ctypes.c_double, ctypes.c_uint64, ctypes.c_void_p]
        L.synth_streams.restype = ctypes.c_int
        L.synth_streams.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64, ctypes.c_void_p,
                                    ctypes.c_int32, ctypes.c_int64, ctypes.c_void_p, ctypes.c_int32,
                                    ctypes.c_void_p, ctypes.c_void_p]
        _lib = L
    return _lib


def splitmix64(x: int) -> int:
    return int(lib().synth_splitmix64(ctypes.c_uint64(x & ((1 << 64) - 1))))


def markov_table(order: int, alpha: float, seed: int) -> np.ndarray:
    n = int(lib().synth_markov_rows(order))
    cdf = np.empty((n, 256), np.float32)
    if lib().synth_markov_table(order, alpha, ctypes.c_uint64(seed), cdf.ctypes.data) != 0:
        raise ValueError("bad markov table arguments")
    return cdf


def zipf_table(s: float, seed: int) -> np.ndarray:
    cdf = np.empty(256, np.float32)
    if lib().synth_zipf_table(s, ctypes.c_uint64(seed), cdf.ctypes.data) != 0:
        raise ValueError("bad zipf arguments")
    return cdf


def cdf_probs(cdf: np.ndarray) -> np.ndarray:
    """Per-symbol probabilities a cumulative table encodes (rows of 256)."""
    c = np.asarray(cdf, np.float64)
    p = np.diff(c, axis=-1, prepend=0.0)
    return p / c[..., -1:]


def generate(sources, src_of: np.ndarray, seg_len: int, L: int, stream_seeds: np.ndarray):
    """Draw B streams of length L.  sources: list of (type, order, cdf-or-None);
    src_of: int32 [B][n_seg] source per segment.  Returns (uint8 [B][L],
    source code length in bits per stream [B])."""
    src_of = np.ascontiguousarray(src_of, np.int32)
    B, n_seg = src_of.shape
    keep = []
    arr = (_Source * len(sources))()
    for i, (typ, order, cdf) in enumerate(sources):
        arr[i].type = typ
        arr[i].order = order
        if cdf is not None:
            c = np.ascontiguousarray(cdf, np.float32)
            keep.append(c)
            arr[i].cdf = c.ctypes.data
        else:
            arr[i].cdf = None
    seeds = np.ascontiguousarray(stream_seeds, np.uint64)
    assert seeds.shape == (B,)
    out = np.empty((B, L), np.uint8)
    codelen = np.zeros(B, np.float64)
    rc = lib().synth_streams(out.ctypes.data, B, L, src_of.ctypes.data, n_seg, seg_len,
                             ctypes.cast(arr, ctypes.c_void_p), len(sources), seeds.ctypes.data,
                             codelen.ctypes.data)
    if rc != 0:
        raise ValueError("synth_streams rejected its arguments")
    return out, codelen


def random_streams(seed: int, B: int, L: int) -> np.ndarray:
    """Uniform random bytes (numpy PCG64), for small tests."""
    return np.random.default_rng(seed).integers(0, 256, size=(B, L), dtype=np.uint8)


def random_windows(seed: int, N: int, W: int):
    """N independent uniform windows and targets (bytes), for small tests."""
    r = np.random.default_rng(seed)
    return (r.integers(0, 256, size=(N, W), dtype=np.uint8),
            r.integers(0, 256, size=N, dtype=np.uint8))


def random_flat(seed: int, n: int, std: float = 0.02) -> np.ndarray:
    """A flat fp32 parameter vector of i.i.d. N(0, std) entries (numpy PCG64)."""
    return (np.random.default_rng(seed).standard_normal(n) * std).astype(np.float32)


def sample_positions(seed: int, B: int, L: int, W: int, n: int):
    """n seeded (stream, target position) pairs with a full window."""
    r = np.random.default_rng(seed)
    return r.integers(0, B, size=n), r.integers(W, L, size=n)


def shared_markov_streams(B: int, L: int, order: int, alpha: float, seed: int):
    """B streams drawn from ONE order-k Markov source with Dirichlet(alpha)
    rows (a context every stream shares, so a shared model can learn it):
    (uint8 [B][L], source code length [B] bits)."""
    src = [(SRC_MARKOV, order, markov_table(order, alpha, splitmix64(seed ^ 0xABCDEF)))]
    seeds = np.array([splitmix64(seed ^ (b + 1)) for b in range(B)], np.uint64)
    return generate(src, np.zeros((B, 1), np.int32), L, L, seeds)


def performer_features(seed: int, m: int, dh: int, orthogonal: bool = True) -> np.ndarray:
    """The random projection of a Performer's positive random features: m
    vectors omega_i in R^dh, i.i.d. N(0, I) or, when orthogonal, rows of
    Gram-Schmidt-orthogonalised Gaussian blocks of dh rows rescaled by the
    norms of independent N(0, I) vectors (orthogonal random features).
    float32 [m][dh]; numpy PCG64 seeded with `seed`."""
    r = np.random.default_rng(seed)
    if not orthogonal:
        return r.standard_normal((m, dh)).astype(np.float32)
    blocks = []
    for _ in range(-(-m // dh)):
        q, _ = np.linalg.qr(r.standard_normal((dh, dh)))
        blocks.append(q.T)
    w = np.concatenate(blocks)[:m]
    norms = np.linalg.norm(r.standard_normal((m, dh)), axis=1)
    return (w * norms[:, None]).astype(np.float32)


from .workloads import workload_streams  # noqa: E402,F401
