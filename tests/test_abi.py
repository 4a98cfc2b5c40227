"""The C ABI without a GPU: the library loads and exports every function that
include/trace.h declares; the host-only calls (parameter count, seeded
initialiser, back-prop controller, configuration checks) agree with the oracle
and return the documented error codes."""
import math
import os
import re

import numpy as np
import pytest

import oracle as O
import paper_2203_16114_amd as P
from synth import WORKLOADS

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "trace.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(trace_[a-z_]+)\s*\(", src)))


def test_library_exports_every_declared_function():
    names = _declared()
    assert len(names) >= 17
    L = P.lib()
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(P.EXPORTS)


@pytest.mark.parametrize("wid", sorted(WORKLOADS))
def test_param_count_matches_oracle(wid):
    w = WORKLOADS[wid]
    cfg = P.make_config(w.W, w.e, w.g, w.H, w.F, w.k, w.dtype)
    assert P.param_count(cfg) == O.param_count(O.Config(W=w.W, e=w.e, g=w.g, H=w.H, F=w.F, k=w.k))


@pytest.mark.parametrize("wid,seed", [(1, 0), (2, 0x7ACE1002), (4, 12345), (5, 2 ** 64 - 1)])
def test_initialiser_is_bit_exact_with_oracle(wid, seed):
    w = WORKLOADS[wid]
    cfg = P.make_config(w.W, w.e, w.g, w.H, w.F, w.k, w.dtype)
    a = P.init_flat_host(cfg, seed, 0.02)
    b = O.init_flat(O.Config(W=w.W, e=w.e, g=w.g, H=w.H, F=w.F, k=w.k), seed, 0.02)
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
    assert np.all(a[-256:] == 0)


def test_controller_is_bit_exact_with_oracle_on_random_sequences():
    r = np.random.default_rng(7)
    for trial in range(40):
        t = int(r.integers(1, 257)) if trial % 4 else int(r.integers(1, 9))
        delta = float(r.choice([0.0, 0.05, -0.01, float(r.uniform(0, 0.2))]))
        n = 2500
        base = r.uniform(0, 8, size=n)
        # inject exact ties with the threshold now and then
        seq = list(base)
        c, o = P.Controller(t, delta), O.Controller(t, delta)
        for i, e in enumerate(seq):
            if i >= t and i % 17 == 0:
                e = o.threshold()
            assert c.decide(e) == o.decide(e), (trial, i)


def test_controller_worked_example_and_errors():
    c = P.Controller(4, 0.05)
    assert [c.decide(x) for x in [8, 7, 6, 5, 5, 5.8, 6, 5]] == [1, 1, 1, 1, 0, 0, 1, 0]
    with pytest.raises(P.TraceError) as ei:
        c.decide(math.nan)
    assert ei.value.code == P.TRACE_ENONFINITE
    assert c.decide(9.0) == 1  # the rejected value did not enter the cache
    for bad_t in (0, 257, -3):
        with pytest.raises(P.TraceError) as ei:
            P.Controller(bad_t, 0.05)
        assert ei.value.code == P.TRACE_EINVAL


@pytest.mark.parametrize("kw", [dict(W=18, g=4), dict(H=3), dict(k=0), dict(k=9), dict(F=0), dict(e=0),
                                dict(dtype=7), dict(beta1=1.0), dict(eps=0.0), dict(max_keep=-1)])
def test_invalid_configs_are_rejected(kw):
    base = dict(W=16, e=16, g=4, H=1, F=256, k=2, dtype="fp32", use_pos=True, max_windows=1024, max_keep=0,
                lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8)
    base.update(kw)
    cfg = P.make_config(**base)
    with pytest.raises(P.TraceError) as ei:
        P.param_count(cfg)
    assert ei.value.code == P.TRACE_EINVAL
    assert P.lib().trace_last_error().decode() != ""


def test_strerror_names_every_code():
    L = P.lib()
    for code in (0, -1, -2, -3, -4, -5, -6):
        assert L.trace_strerror(code).decode() not in ("", "unknown error")
    assert L.trace_strerror(-99).decode() == "unknown error"


@pytest.mark.parametrize("wid,seed", [(2, 3), (4, 77)])
def test_untied_layout_and_initialiser_match_oracle(wid, seed):
    w = WORKLOADS[wid]
    cfg = P.make_config(w.W, w.e, w.g, w.H, w.F, w.k, w.dtype, untied_ffn=True)
    ocf = O.Config(W=w.W, e=w.e, g=w.g, H=w.H, F=w.F, k=w.k, untied=True)
    assert P.param_count(cfg) == O.param_count(ocf)
    a = P.init_flat_host(cfg, seed, 0.02)
    b = O.init_flat(ocf, seed, 0.02)
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))


@pytest.mark.parametrize("layers,untied", [(2, False), (3, True)])
def test_multilayer_layout_and_init_match_oracle(layers, untied):
    w = WORKLOADS[4]
    cfg = P.make_config(w.W, w.e, w.g, w.H, w.F, w.k, w.dtype, untied_ffn=untied, layers=layers)
    ocfg = O.Config(W=w.W, e=w.e, g=w.g, H=w.H, F=w.F, k=w.k, untied=untied, layers=layers)
    assert P.param_count(cfg) == O.param_count(ocfg)
    a = P.init_flat_host(cfg, 77)
    b = O.init_flat(ocfg, 77)
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
