"""GPU parity of the coding: the quantisation kernel bit for bit against the
coding oracle, and the compressor of Alg. 1 (forward -> frequencies -> range
code -> controller -> update) decoding back to its input with the same
updates, on the shapes of the workloads."""
import numpy as np
import pytest

import oracle as O
import oracle.coder as C
import synth
from gpu_helpers import make_model, ocfg, to_dev, workload_cfg

pytestmark = pytest.mark.gpu


def _logits(seed, n):
    rng = np.random.default_rng(seed)
    z = (rng.standard_normal((n, 256)) * rng.uniform(0.05, 20, (n, 1))).astype(np.float32)
    z[::7, :] = np.round(z[::7, :])                      # ties
    z[3::11, :] = 0.0                                    # uniform rows
    z[5::13, 17] = 80.0                                  # one dominant byte, others below 2^-32
    return z


@pytest.mark.parametrize("n", [1, 3, 4, 1021, 4099])
def test_quantize_bit_exact(n):
    import torch
    import paper_2203_16114_amd as P
    z = _logits(n, n)
    f = P.quantize(to_dev(z))
    torch.cuda.synchronize()
    got = f.cpu().numpy().view(np.uint16).astype(np.int64)
    assert np.array_equal(got, C.quantize(z))


def test_quantize_empty_is_a_no_op():
    import torch
    import paper_2203_16114_amd as P
    z = torch.zeros(0, 256, dtype=torch.float32, device="cuda")
    assert P.quantize(z).numel() == 0


@pytest.mark.parametrize("mode", [C.MODE_NEVER, C.MODE_GATED, C.MODE_ALWAYS])
def test_round_trip_adaptation_shape(mode):
    """bf16 model of the adaptation workload's shape (d=128, T=8), 48 streams:
    the decoder rebuilds every byte, takes the same updates and ends with the
    same weights."""
    shape, dtype = workload_cfg(4)
    streams, _ = synth.workload_streams(4, L=160, B=48)
    enc = make_model(shape, dtype, seed=5, max_windows=64, max_keep=64)
    dec = make_model(shape, dtype, seed=5, max_windows=64, max_keep=64)
    codes, nu = enc.compress(to_dev(streams), mode=mode, t=4, delta=0.0)
    out, nu2 = dec.decompress(codes, 160, mode=mode, t=4, delta=0.0)
    assert np.array_equal(out.cpu().numpy(), streams)
    assert nu == nu2
    if mode == C.MODE_ALWAYS:
        assert nu == 160 - shape["W"]
    if mode == C.MODE_NEVER:
        assert nu == 0
    if mode == C.MODE_GATED:
        assert 0 < nu < 160 - shape["W"]
    te, me, ve, se = enc.get_state()
    td, md, vd, sd = dec.get_state()
    assert se == sd and np.array_equal(te, td) and np.array_equal(me, md)


def test_code_length_matches_estimated_bits_main_shape():
    """Without updates a stream's code is its estimated bits (the headline
    quantity) plus the quantisation and a few bytes: within 0.5 % + 8 bytes."""
    import torch
    shape, dtype = workload_cfg(3)
    L = 64 + 300
    streams, _ = synth.workload_streams(3, L=L, B=32)
    m = make_model(shape, dtype, seed=8, max_windows=1 << 14)
    codes, _ = m.compress(to_dev(streams))
    r = m.forward_bits(to_dev(streams), 64, L - 64)
    torch.cuda.synchronize()
    bits = r["bits"].view(32, L - 64).double().sum(1).cpu().numpy() + 64 * 8
    size = np.array([8 * len(c) for c in codes], np.float64)
    assert np.all(np.abs(size - bits) <= 0.005 * bits + 64)
    out, _ = make_model(shape, dtype, seed=8, max_windows=1 << 14).decompress(codes, L)
    assert np.array_equal(out.cpu().numpy(), streams)


def test_fp32_codes_close_to_oracle_codes():
    """Tiny fp32 model: the library's code lengths against the coding oracle's
    (fp64 model, the same quantisation and coder) on the same streams."""
    shape = dict(W=16, e=16, g=4, H=1, F=256, k=2)
    streams = synth.random_streams(3, 6, 120)
    flat = O.init_flat(ocfg(**shape), 21)
    m = make_model(shape, "fp32", seed=0, flat=flat)
    codes, _ = m.compress(to_dev(streams))
    ref, _ = C.compress(flat, ocfg(**shape), streams)
    for a, b in zip(codes, ref):
        assert abs(len(a) - len(b)) <= 0.002 * len(b) + 2
    out, _ = make_model(shape, "fp32", seed=0, flat=flat).decompress(codes, 120)
    assert np.array_equal(out.cpu().numpy(), streams)


def test_short_streams_and_errors():
    import paper_2203_16114_amd as P
    shape = dict(W=16, e=16, g=4, H=1, F=256, k=2)
    s = synth.random_streams(4, 3, 10)                  # shorter than the window: all at 1/256
    m = make_model(shape, "fp32", seed=1)
    codes, nu = m.compress(to_dev(s))
    assert nu == 0 and all(c == C.encode_symbols([C.UNIFORM] * 10, list(r)) for c, r in zip(codes, s))
    out, _ = make_model(shape, "fp32", seed=1).decompress(codes, 10)
    assert np.array_equal(out.cpu().numpy(), s)
    with pytest.raises(P.TraceError):                    # updates need max_keep >= streams
        m.compress(to_dev(synth.random_streams(4, 3, 40)), mode=C.MODE_GATED)


def test_round_trip_large_shape_gated():
    """The large mixed workload's shape (d=512, e=64, W=64, F=2048, k=3, bf16),
    64 streams, controller-gated: every byte back, the same updates and the
    same final weights."""
    shape, dtype = workload_cfg(5)
    L = 64 + 40
    streams, _ = synth.workload_streams(5, L=L, B=64)
    enc = make_model(shape, dtype, seed=2, max_windows=64, max_keep=64)
    dec = make_model(shape, dtype, seed=2, max_windows=64, max_keep=64)
    codes, nu = enc.compress(to_dev(streams), mode=C.MODE_GATED, t=4, delta=0.0)
    out, nu2 = dec.decompress(codes, L, mode=C.MODE_GATED, t=4, delta=0.0)
    assert np.array_equal(out.cpu().numpy(), streams) and nu == nu2 and nu >= 4
    assert np.array_equal(enc.get_state()[0], dec.get_state()[0])


def test_strided_streams():
    """Rows longer than the coded length (the encoder packs them on the device;
    the decoder writes into wider rows): the same codes as the packed layout."""
    import torch
    shape = dict(W=16, e=16, g=4, H=1, F=256, k=2)
    s = synth.random_streams(8, 700, 90)                 # 700 streams: the threaded coding path
    wide = np.concatenate([s, np.full((700, 13), 0xAB, np.uint8)], axis=1)
    a, _ = make_model(shape, "fp32", seed=3, max_windows=1024, max_keep=1024).compress(
        to_dev(wide), mode=C.MODE_ALWAYS, length=90)
    b, _ = make_model(shape, "fp32", seed=3, max_windows=1024, max_keep=1024).compress(
        to_dev(s), mode=C.MODE_ALWAYS)
    assert a == b
    out = torch.full((700, 103), 7, dtype=torch.uint8, device="cuda")
    got, nu = make_model(shape, "fp32", seed=3, max_windows=1024, max_keep=1024).decompress(
        a, 90, mode=C.MODE_ALWAYS, out=out)
    o = out.cpu().numpy()
    assert np.array_equal(o[:, :90], s) and np.all(o[:, 90:] == 7) and nu == 90 - 16
