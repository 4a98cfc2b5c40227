"""The library's host side of the coding (the 2^(-j/256) table and the range
coder) against the coding oracle, bit for bit: CPU only, no GPU calls."""
import itertools

import numpy as np
import pytest

import oracle.coder as C


@pytest.fixture(scope="module")
def P():
    import paper_2203_16114_amd as P
    return P


def test_table_equals_oracle(P):
    assert np.array_equal(P.quant_table().astype(np.int64), np.array(C.quant_table(), np.int64))


@pytest.mark.parametrize("seed,n,scale", [(1, 1, 1.0), (2, 257, 3.0), (3, 2000, 12.0)])
def test_codes_equal_oracle(P, seed, n, scale):
    rng = np.random.default_rng(seed)
    z = (rng.standard_normal((n, 256)) * scale).astype(np.float32)
    F = C.quantize(z)
    x = [int(rng.choice(256, p=r / r.sum())) for r in F]
    code = P.rc_encode(F.astype(np.uint16), x)
    assert code == C.encode_symbols(F, x)
    assert list(P.rc_decode(F.astype(np.uint16), code, n)) == x


def test_uniform_and_carry_codes_equal_oracle(P):
    rng = np.random.default_rng(9)
    x = list(rng.integers(0, 256, 500))
    assert P.rc_encode(None, x) == C.encode_symbols([C.UNIFORM] * 500, x)
    # symbols at the top of the interval: carries through held-back 0xFF bytes
    F = np.ones((3000, 256), np.uint16)
    F[:, 255] = 65536 - 255
    y = [255] * 2999 + [0]
    code = P.rc_encode(F, y)
    assert code == C.encode_symbols(F.astype(np.int64), y)
    assert list(P.rc_decode(F, code, 3000)) == y


def test_brute_force_short_sequences(P):
    F = np.ones((4, 256), np.uint16)
    F[:, :3] = [[1, 2, 5]] * 4
    for seq in itertools.product(range(3), repeat=4):
        code = P.rc_encode(F, list(seq))
        assert code == C.encode_symbols(F.astype(np.int64), list(seq))
        assert tuple(P.rc_decode(F, code, 4)) == seq


def test_empty_and_errors(P):
    assert P.rc_encode(None, []) == C.encode_symbols([], [])
    assert len(P.rc_decode(None, b"", 0)) == 0
    bad = np.ones((1, 256), np.uint16)
    bad[0, 7] = 0
    with pytest.raises(P.TraceError):
        P.rc_encode(bad, [7])
    big = np.full((1, 256), 300, np.uint16)          # total 76800 > 65536
    with pytest.raises(P.TraceError):
        P.rc_decode(big, b"\0\0\0\0\0", 1)
