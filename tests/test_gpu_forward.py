"""Forward parity of the HIP path (through the C ABI) against the CPU oracle.

Inputs are the seeded synthetic streams of the five workloads (prefixes of
them where the full size is not needed) and weights from the shared seeded
initialiser.  fp32 models are compared with the oracle in fp64, bf16 models
with the oracle emulating the bf16 storage points."""
import numpy as np
import pytest
import torch

import oracle as O
import synth
from gpu_helpers import check_parity, make_model, ocfg, oracle_mode, structured_flat, to_dev, workload_cfg

pytestmark = pytest.mark.gpu


def _oracle_at(shape, flat, streams, b, i, mode, use_pos=True):
    cfg = ocfg(**shape, use_pos=use_pos)
    w, y = O.windows_at(streams, b, i, cfg.W)
    return O.forward(flat, cfg, w, y, mode=mode)


# ------------------------------------------- byte-group indexing, bit-exact
_INDEX_CASES = [(1, "fp32"), (2, "fp32"), (3, "bf16"), (4, "bf16"), (5, "bf16"), (4, "fp32")]


@pytest.mark.parametrize("wid,dtype", _INDEX_CASES)
def test_byte_group_indexing_is_bit_exact_in_the_forward_kernels(wid, dtype):
    """The gathers inside the path's kernels: the per-token attention kernel at
    both tile sizes (launch sizes below and above the chip-filling bound) and,
    in bf16, the shared-group kernel (64-window tiles in one stream, g = 4 and
    8) and the kept-activation variant.  Logits equal the index formula and the
    oracle's bit for bit, for every window."""
    shape, _ = workload_cfg(wid)
    cfg = ocfg(**shape)
    W, T, H = cfg.W, cfg.T, cfg.H
    streams = synth.random_streams(90 + wid, 512, W + 300)
    s = to_dev(streams)
    for r in range(-(-T // H)):
        sel = [(r * H + h) % T for h in range(H)]
        flat, expected = structured_flat(cfg, sel)
        m = make_model(shape, dtype, seed=0, flat=flat, max_windows=1 << 17, max_keep=512)
        launches = [dict(B=3, pos0=W + 11, n=5, kw={}),                       # small tiles
                    dict(B=256, pos0=W + 1, n=256, kw={"token_attn": True}),  # wide tiles
                    dict(B=512, pos0=W + 7, n=1, kw={"keep": True})]          # kept activations
        if dtype == "bf16":
            launches.append(dict(B=256, pos0=W + 3, n=256, kw={}))            # shared byte groups
        for L in launches:
            st = s[:L["B"]].contiguous()
            out = m.forward_bits(st, L["pos0"], L["n"], logits=True, **L["kw"])
            z = out["logits"].cpu().numpy()
            bb, ii = np.meshgrid(np.arange(L["B"]), L["pos0"] + np.arange(L["n"]), indexing="ij")
            win, y = O.windows_at(streams, bb.ravel(), ii.ravel(), W)
            want = expected(win)
            assert np.array_equal(z.view(np.uint32), want.view(np.uint32)), (L, np.argwhere(z != want)[:5])
            pick = np.random.default_rng(r).choice(len(win), size=min(64, len(win)), replace=False)
            ref = O.forward(flat, cfg, win[pick], y[pick], mode=oracle_mode(dtype))
            assert np.array_equal(np.asarray(ref["z"], np.float32).view(np.uint32), want[pick].view(np.uint32))


@pytest.mark.parametrize("wid,dtype", [(1, "fp32"), (2, "fp32"), (3, "bf16"), (4, "bf16"), (5, "bf16")])
def test_update_gather_is_bit_exact(wid, dtype):
    """The update's own gather (the kernel trace_adapt_step runs on the window
    bytes the attention kernel kept) against the oracle's grouping of the
    rounded embedding, bit for bit, over a kept batch with a ragged end."""
    shape, _ = workload_cfg(wid)
    B = 777
    m = make_model(shape, dtype, seed=5, max_keep=B)
    streams = synth.random_streams(11, B, 300)
    pos = shape["W"] + 100
    m.forward_bits(to_dev(streams), pos, 1, keep=True)
    X = m.debug_kept_tokens(B).cpu().numpy()
    cfg = ocfg(**shape, use_pos=False)
    flat = O.init_flat(ocfg(**shape), 5)
    mode = "fp32" if dtype == "fp32" else "bf16"
    p = O.compute_params(flat, ocfg(**shape), mode)
    w, _ = O.windows_at(streams, np.arange(B), np.full(B, pos), cfg.W)
    Xref = O.embed_group(p, w, cfg, O.trace_oracle._Mode(mode)).astype(np.float32)
    if dtype == "bf16":
        got = (X.astype(np.uint16).astype(np.uint32) << 16).view(np.float32)
    else:
        got = X
    assert np.array_equal(got.reshape(Xref.shape).view(np.uint32), Xref.view(np.uint32))


def test_workload1_every_window():
    """Workload 1 (tiny fp32) in full: 16 streams x 4080 windows."""
    shape, dtype = workload_cfg(1)
    streams, _ = synth.workload_streams(1)
    m = make_model(shape, dtype, seed=0x7ACE1001)
    B, L = streams.shape
    W = shape["W"]
    out = m.forward_bits(to_dev(streams), W, L - W, logits=True, step_ce=True)
    bits = out["bits"].cpu().numpy()
    z = out["logits"].cpu().numpy()
    flat = O.init_flat(ocfg(**shape), 0x7ACE1001)
    cfg = ocfg(**shape)
    w, y = O.all_windows(streams, W)
    ref = O.forward(flat, cfg, w, y, mode="fp64")
    check_parity(dtype, z, bits, ref)
    ce = out["step_ce"].cpu().numpy()
    np.testing.assert_allclose(ce, bits.reshape(B, L - W).astype(np.float64).mean(0), rtol=0, atol=1e-12)


@pytest.mark.parametrize("wid,L,B", [(2, 4096, 512), (3, 2048, 4096), (4, 2048, 4096), (5, 1024, 8192)])
def test_workload_sampled_windows(wid, L, B):
    """Every window of a prefix of the workload's streams on the GPU; 2048 seeded
    windows of the result compared with the oracle one by one."""
    shape, dtype = workload_cfg(wid)
    streams, _ = synth.workload_streams(wid, L=L, B=B)
    seed = 0x7ACE1000 + wid
    m = make_model(shape, dtype, seed=seed, max_windows=1 << 18)
    W = shape["W"]
    n_steps = L - W
    out = m.forward_bits(to_dev(streams), W, n_steps, logits=True)
    torch.cuda.synchronize()
    b, i = synth.sample_positions(100 + wid, B, L, W, 2048)
    idx = b * n_steps + (i - W)
    bits = out["bits"][torch.from_numpy(idx).cuda()].cpu().numpy()
    z = out["logits"][torch.from_numpy(idx).cuda()].cpu().numpy()
    flat = O.init_flat(ocfg(**shape), seed)
    ref = _oracle_at(shape, flat, streams, b, i, oracle_mode(dtype))
    check_parity(dtype, z, bits, ref)
    assert np.all(np.isfinite(out["bits"].cpu().numpy()))


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_ragged_tiles_and_chunking_are_bitwise_invariant(dtype):
    """Window counts that leave partial tiles, and a forward split into small
    chunks, give the same bits bit for bit as one launch over everything."""
    shape = dict(W=32, e=32, g=4, H=4, F=512, k=2)
    streams = synth.random_streams(3, 37, 200)
    n_steps = 200 - 32 - 1
    big = make_model(shape, dtype, seed=9, max_windows=1 << 16)
    small = make_model(shape, dtype, seed=9, max_windows=999)
    s = to_dev(streams)
    a = big.forward_bits(s, 32, n_steps, logits=True)
    c = small.forward_bits(s, 32, n_steps, logits=True)
    assert torch.equal(a["bits"], c["bits"]) and torch.equal(a["logits"], c["logits"])
    # one stream, one step: the smallest batch
    d = big.forward_bits(s[5:6].contiguous(), 32 + 17, 1)
    assert torch.equal(d["bits"][0], a["bits"][5 * n_steps + 17])
    flat = O.init_flat(ocfg(**shape), 9)
    bb, ii = np.meshgrid(np.arange(37), 32 + np.arange(n_steps), indexing="ij")
    ref = _oracle_at(shape, flat, streams, bb.ravel(), ii.ravel(), oracle_mode(dtype))
    check_parity(dtype, a["logits"].cpu().numpy(), a["bits"].cpu().numpy(), ref)


@pytest.mark.parametrize("shape", [dict(W=32, e=32, g=4, H=4, F=512, k=2), dict(W=64, e=32, g=8, H=8, F=256, k=1),
                                   dict(W=32, e=32, g=8, H=8, F=256, k=1)])
def test_shared_group_and_token_paths_agree(shape):
    """bf16 launches whose 64-window tiles lie in one stream share the byte groups
    between windows (k_attn_grp; k_attn_wh at d = 256 with 8 heads and g = 8).  A model whose chunks do not start on 64-window
    boundaries runs the token kernel (k_attn) on its later chunks; both match the
    oracle on every window and each other within the bf16 parity bar."""
    W = shape["W"]
    n_steps = 128
    streams = synth.random_streams(21, 9, W + n_steps + 1)
    s = to_dev(streams)
    grp = make_model(shape, "bf16", seed=13, max_windows=1 << 16)
    tok = make_model(shape, "bf16", seed=13, max_windows=65)
    a = grp.forward_bits(s, W, n_steps, logits=True)
    b = tok.forward_bits(s, W, n_steps, logits=True)
    flat = O.init_flat(ocfg(**shape), 13)
    bb, ii = np.meshgrid(np.arange(9), W + np.arange(n_steps), indexing="ij")
    ref = _oracle_at(shape, flat, streams, bb.ravel(), ii.ravel(), oracle_mode("bf16"))
    check_parity("bf16", a["logits"].cpu().numpy(), a["bits"].cpu().numpy(), ref)
    check_parity("bf16", b["logits"].cpu().numpy(), b["bits"].cpu().numpy(), ref)
    za, zb = a["logits"].cpu().numpy(), b["logits"].cpu().numpy()
    rel = np.abs(za - zb).max(axis=1) / np.maximum(np.abs(zb).max(axis=1), 1e-6)
    assert rel.max() < 2e-2


def test_permuting_streams_permutes_outputs_bitwise():
    shape, dtype = workload_cfg(3)
    streams, _ = synth.workload_streams(3, L=400, B=96)
    perm = np.random.default_rng(4).permutation(96)
    m = make_model(shape, dtype, seed=77)
    a = m.forward_bits(to_dev(streams), 64, 400 - 64)["bits"].view(96, -1)
    b = m.forward_bits(to_dev(streams[perm]), 64, 400 - 64)["bits"].view(96, -1)
    assert torch.equal(a[torch.from_numpy(perm).cuda()], b)


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_zeroed_head_gives_exactly_8_bits(dtype):
    shape = dict(W=16, e=16, g=4, H=1, F=256, k=2)
    cfg = ocfg(**shape)
    flat = O.init_flat(cfg, 21)
    p = O.unflatten(flat, cfg)
    p["Wout"][:] = 0
    p["bout"][:] = 0
    m = make_model(shape, dtype, seed=0, flat=flat)
    streams = synth.random_streams(8, 5, 100)
    bits = m.forward_bits(to_dev(streams), 16, 84)["bits"].cpu().numpy()
    assert np.all(bits == 8.0)


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_without_positional_table(dtype):
    shape = dict(W=32, e=32, g=4, H=4, F=512, k=2)
    m = make_model(shape, dtype, seed=13, use_pos=False)
    streams = synth.random_streams(6, 9, 300)
    out = m.forward_bits(to_dev(streams), 32, 268, logits=True)
    cfg = ocfg(**shape, use_pos=False)
    flat = O.init_flat(cfg, 13)
    w, y = O.all_windows(streams, 32, 32, 268)
    ref = O.forward(flat, cfg, w, y, mode=oracle_mode(dtype))
    check_parity(dtype, out["logits"].cpu().numpy(), out["bits"].cpu().numpy(), ref)


def test_argument_errors_and_empty_batches():
    import paper_2203_16114_amd as P
    shape = dict(W=16, e=16, g=4, H=1, F=256, k=2)
    m = make_model(shape, "fp32", seed=1)
    s = to_dev(synth.random_streams(1, 2, 64))
    with pytest.raises(P.TraceError) as ei:
        m.forward_bits(s, 15, 4)           # pos0 < W
    assert ei.value.code == P.TRACE_EINVAL
    with pytest.raises(P.TraceError) as ei:
        m.forward_bits(s, 16, 4, keep=True)  # model built without max_keep
    assert ei.value.code == P.TRACE_EINVAL
    with pytest.raises(P.TraceError) as ei:
        m.adapt_step()
    assert ei.value.code == P.TRACE_ESTATE
    out = m.forward_bits(s, 16, 0)
    assert out["bits"].numel() == 0
    with pytest.raises(P.TraceError) as ei:
        P.TraceModel(W=24, e=16, g=4, H=1, F=256, k=2)  # T = 6 has no kernel
    assert ei.value.code == P.TRACE_EUNSUPPORTED
