"""Pins of the coding oracle (oracle/coder.py) against closed forms, exact
integer characterisations, invariants and brute force: CPU only."""
import itertools
import math

import numpy as np
import pytest

from oracle import coder as C
import oracle as O


def test_quant_table_is_correctly_rounded():
    # T[j] = round(2^31 2^(-j/256)) iff (2T-1)^256 < 2^256 2^(31*256-j) < (2T+1)^256:
    # exact integer comparisons, independent of the decimal arithmetic
    T = C.quant_table()
    assert T[0] == 2 ** 31 and T[128] == 1518500250
    for j, t in enumerate(T):
        mid = 2 ** 256 * 2 ** (31 * 256 - j)
        assert (2 * t - 1) ** 256 < mid < (2 * t + 1) ** 256, j
    assert all(a > b for a, b in zip(T, T[1:]))


def test_quantize_closed_forms():
    z = np.zeros((1, 256), np.float32)
    assert np.all(C.quantize(z) == 256)                    # uniform: 1 + 65280/256
    z = np.full((1, 256), -100.0, np.float32)
    z[0, 77] = 3.0
    f = C.quantize(z)[0]                                   # one byte takes the spread
    assert f[77] == 1 + 65280 and np.all(np.delete(f, 77) == 1)
    z = np.zeros((1, 256), np.float32)
    z[0, 128:] = -np.float32(math.log(2.0))                # weights 2^31 and 2^30
    f = C.quantize(z)[0]
    assert np.all(f[:128] == 1 + 65280 * 2 // 384) and np.all(f[128:] == 1 + 65280 // 384)


def test_quantize_invariants():
    rng = np.random.default_rng(3)
    z = (rng.standard_normal((200, 256)) * rng.uniform(0.1, 8, (200, 1))).astype(np.float32)
    f = C.quantize(z)
    tot = f.sum(1)
    assert f.min() >= 1 and tot.max() <= 65536 and tot.min() >= 65536 - 256
    # monotone in the logit, and close to the softmax
    order = np.argsort(z, axis=1)
    assert np.all(np.diff(np.take_along_axis(f, order, 1), axis=1) >= 0)
    p = np.exp(z - z.max(1, keepdims=True)); p /= p.sum(1, keepdims=True)
    # 1 - 65280/65536 of each share is reserved for the minimum frequency
    # (0.39 %), and a weight is off by at most a step of 2^(1/256) (0.14 %)
    assert np.all(np.abs(f / tot[:, None] - p) <= 0.006 * p + 3.0 / 65536)
    # shift invariance of the logits that keep the float32 differences exact
    assert np.array_equal(C.quantize(z), C.quantize(z + np.float32(0.0)))


def test_range_coder_round_trip_and_length():
    rng = np.random.default_rng(5)
    for n in (1, 7, 300):
        z = (rng.standard_normal((n, 256)) * 3).astype(np.float32)
        F = C.quantize(z)
        x = [int(rng.choice(256, p=r / r.sum())) for r in F]
        code = C.encode_symbols(F, x)
        assert code[0] == 0
        assert C.decode_symbols(F, code) == x
        ideal = sum(C.coded_bits(F[i], x[i]) for i in range(n))
        assert ideal - 8 <= 8 * len(code) <= ideal + 48
    u = [C.UNIFORM] * 100
    x = list(rng.integers(0, 256, 100))
    code = C.encode_symbols(u, x)
    assert C.decode_symbols(u, code) == x and len(code) <= 100 + 6


def test_range_coder_brute_force_small_alphabets():
    # every sequence of length <= 5 over three symbols of frequencies (1, 2, 5),
    # and (1, 65534, 1) at the largest total: decodes to itself, codes distinct
    for freqs in ([1, 2, 5], [1, 65534, 1]):
        for n in range(1, 6):
            seen = {}
            for seq in itertools.product(range(3), repeat=n):
                code = C.encode_symbols([freqs] * n, seq)
                assert C.decode_symbols([freqs] * n, code) == list(seq)
                assert code not in seen
                seen[code] = seq


def test_range_coder_carry():
    # symbols at the top of the interval drive low past 2^32: the carry must
    # reach the bytes already held back
    F = [[1, 65535]] * 2000
    x = [1] * 1999 + [0]
    code = C.encode_symbols(F, x)
    assert C.decode_symbols(F, code) == x


@pytest.mark.parametrize("mode", [C.MODE_NEVER, C.MODE_GATED, C.MODE_ALWAYS])
def test_compress_round_trip_tiny(mode):
    cfg = O.Config(W=16, e=16, g=4, H=1, F=64, k=1)
    flat = O.init_flat(cfg, 4)
    rng = np.random.default_rng(11)
    streams = rng.integers(0, 8, (3, 28)).astype(np.uint8)    # a small alphabet: compressible
    codes, dec = C.compress(flat, cfg, streams, mode=mode, t=2, delta=0.0)
    out, dec2 = C.decompress(flat, cfg, codes, 28, mode=mode, t=2, delta=0.0)
    assert np.array_equal(out, streams) and dec == dec2
    assert len(dec) == 28 - 16
    if mode == C.MODE_ALWAYS:
        assert all(dec)
    if mode == C.MODE_NEVER:
        assert not any(dec)
        # the coded length matches the model's code length within quantisation
        w, y = O.windows_at(streams, np.repeat(np.arange(3), 12), np.tile(np.arange(16, 28), 3), 16)
        bits = O.forward(flat, cfg, w, y)["bits"].reshape(3, 12).sum(1) + 16 * 8
        for b in range(3):
            assert 8 * len(codes[b]) <= bits[b] * 1.01 + 48
