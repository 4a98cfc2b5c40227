"""The five workloads: model shape, precision, mode and byte-stream recipe.

Shapes follow the paper's model family (Sec. 4: byte-grouping, one attention
layer, a shared FFN; Sec. 6 trains with Adam at lr 1e-3 from a random start)
scaled to the sizes benchmarked here.  Stream recipes are seeded; the seeds are
0x7ACE0000 + id for the streams and 0x7ACE1000 + id for the weights.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np


@dataclass(frozen=True)
class Workload:
    id: int
    name: str
    B: int          # independent streams (one window each per step)
    L: int          # bytes per stream
    W: int          # window bytes
    e: int          # per-byte embedding width
    g: int          # bytes per group (token)
    H: int          # heads
    F: int          # FFN width
    k: int          # shared-FFN repeats
    dtype: str      # "fp32" or "bf16" (bf16 operands, fp32 accumulate + master)
    mode: str       # "fwd" (forward + bits) or "gated" (controller-gated adaptation)
    t: int = 16     # controller cache size
    delta: float = 0.05  # controller margin, bits

    @property
    def T(self):
        return self.W // self.g

    @property
    def d(self):
        return self.g * self.e

    @property
    def stream_seed(self):
        return 0x7ACE0000 + self.id

    @property
    def weight_seed(self):
        return 0x7ACE1000 + self.id


WORKLOADS = {
    1: Workload(1, "tiny-fp32", 16, 4096, 16, 16, 4, 1, 256, 2, "fp32", "fwd"),
    2: Workload(2, "small-fp32", 512, 65536, 32, 32, 4, 4, 512, 2, "fp32", "fwd"),
    3: Workload(3, "main-bf16", 4096, 262144, 64, 32, 8, 8, 1024, 3, "bf16", "fwd"),
    4: Workload(4, "adapt-bf16", 4096, 32768, 32, 32, 4, 4, 512, 2, "bf16", "gated"),
    5: Workload(5, "large-mixed-bf16", 8192, 262144, 64, 64, 8, 8, 2048, 3, "bf16", "gated"),
}

# regime length for workload 4: 8 MiB of batch input between source switches
# = 2048 bytes per stream at B = 4096
REGIME_BYTES_PER_STREAM = 2048


def _stream_seeds(base: int, B: int):
    from . import splitmix64
    return np.array([splitmix64(base ^ (b + 1)) for b in range(B)], np.uint64)


def _table_seed(base: int, src_id: int):
    from . import splitmix64
    return splitmix64(base ^ 0xABCDEF ^ src_id)


def workload_streams(wid: int, L: int | None = None, B: int | None = None):
    """Streams of workload wid: (uint8 [B][L], source code length [B] bits).
    L (and B) may be cut short; a shorter L gives a prefix of the full streams
    and a smaller B the first B of them."""
    from . import (SRC_MARKOV, SRC_RUNS, SRC_UNIFORM, SRC_ZIPF, generate,
                   markov_table, zipf_table)
    w = WORKLOADS[wid]
    L = w.L if L is None else int(L)
    Bfull = w.B
    B = Bfull if B is None else int(B)
    base = w.stream_seed
    seeds = _stream_seeds(base, Bfull)[:B]
    rng = np.random.default_rng(base)
    if wid == 1:
        src = [(SRC_MARKOV, 1, markov_table(1, 0.1, _table_seed(base, 0)))]
        of = np.zeros((Bfull, 1), np.int32)
        seg = L
    elif wid == 2:
        src = [(SRC_MARKOV, 2, markov_table(2, 0.05, _table_seed(base, 0))),
               (SRC_ZIPF, 0, zipf_table(1.1, _table_seed(base, 1)))]
        of = (np.arange(Bfull) >= Bfull // 2).astype(np.int32)[:, None]
        seg = L
    elif wid == 3:
        src = [(SRC_MARKOV, 3, markov_table(3, 0.02, _table_seed(base, 0))),
               (SRC_ZIPF, 0, zipf_table(1.2, _table_seed(base, 1))),
               (SRC_UNIFORM, 0, None)]
        of = (np.arange(Bfull) % 3).astype(np.int32)[:, None]
        seg = L
    elif wid == 4:
        seg = REGIME_BYTES_PER_STREAM
        n_reg = max(1, -(-L // seg))
        pairs, prev = [], None
        orders, alphas = (1, 2, 3), (0.02, 0.05, 0.2, 1.0)
        for _ in range(n_reg):
            while True:
                pr = (orders[rng.integers(3)], alphas[rng.integers(4)])
                if pr != prev:
                    break
            pairs.append(pr)
            prev = pr
        src = [(SRC_MARKOV, o, markov_table(o, a, _table_seed(base, r)))
               for r, (o, a) in enumerate(pairs)]
        of = np.tile(np.arange(n_reg, dtype=np.int32)[None, :], (Bfull, 1))
    elif wid == 5:
        n_mk = 12
        mk = [(int(rng.integers(1, 5)), (0.01, 0.1, 1.0)[rng.integers(3)]) for _ in range(n_mk)]
        kind = rng.permutation(np.repeat(np.arange(4), Bfull // 4))  # 0 markov 1 zipf 2 unif 3 runs
        mk_pick = rng.integers(0, n_mk, size=Bfull)
        zs = rng.uniform(1.0, 1.5, size=Bfull)
        src = [(SRC_MARKOV, o, markov_table(o, a, _table_seed(base, i))) for i, (o, a) in enumerate(mk)]
        src += [(SRC_UNIFORM, 0, None), (SRC_RUNS, 0, None)]
        of = np.zeros((Bfull, 1), np.int32)
        for b in range(B):
            if kind[b] == 0:
                of[b, 0] = mk_pick[b]
            elif kind[b] == 1:
                src.append((SRC_ZIPF, 0, zipf_table(float(zs[b]), _table_seed(base, 1000 + b))))
                of[b, 0] = len(src) - 1
            elif kind[b] == 2:
                of[b, 0] = n_mk
            else:
                of[b, 0] = n_mk + 1
        seg = L
    else:
        raise KeyError(wid)
    return generate(src, of[:B], seg, L, seeds)
