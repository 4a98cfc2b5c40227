#!/usr/bin/env python3
"""Throughput of TRACE's batched next-byte estimator on one MI355X.

A step is one call of the forward estimator with code lengths over a batch of
windows of the main workload (4096 streams, W = 64 bytes, e = 32, g = 8 -> 8
tokens of d = 256, 8 heads, FFN 1024 shared x3, bf16 operands with fp32
accumulation): `--steps-per-call` consecutive positions of every stream, i.e.
4096 x S windows.  Successive steps walk along the streams.  The value is
predicted bytes (= windows) per second over the timed steps, with the streams
already in device memory.

Besides the headline line this run measures:
  - the forward of the tiny and small fp32 workloads and of the large bf16
    workload (bytes/s and the fraction of the MFMA peak of their dtype);
  - the controller-gated loop of Alg. 1 / Alg. 2 (trace_gated_run) against the
    always-update loop on the adaptation workload (its whole 32 KiB streams,
    16 source regimes) and on the large mixed workload (4096 steps), with the
    configured margin (0.05 bits) and with Eq. 7's margin 0;
  - the compressor / decompressor round trip, the deep-FFN variant;
  - the CPU oracle on a bounded sample of the main workload's windows, on all
    host cores and on one.

Prints ONE JSON line (rank 0).  Only one GPU is supported.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_TFLOPS = {"bf16": 2500.0, "fp32": 157.3}   # MI355X dense MFMA peaks
HBM_GBS = 8000.0


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def flops_per_window(w):
    """Algorithmic flops of the last-token readout path, split by kernel:
    attention block 4*T*d^2 (K, V of all T tokens) + 2*d^2 (q) + 2*d^2 (Wo)
    + 4*T*d (scores, weighted values); FFN+head 4*k*d*F + 512*d."""
    T, d, F, k = w.T, w.d, w.F, w.k
    return {"attn": 4 * T * d * d + 4 * d * d + 4 * T * d, "ffn_head": 4 * k * d * F + 512 * d}


def mfma_flops_per_window(w):
    """Flops the matrix cores execute per window on the main workload's launches
    (bf16, 64-window tiles within one stream): the attention block projects the
    tile's 128 byte-group rows (the 120 distinct groups of its 64 windows, in
    16-row fragments) to K and V once, 128 * 4d^2 / 64 = 8d^2 per window, plus
    q and Wo (2d^2 each); the scores and weighted sums run on the vector ALUs.
    The FFN executes its algorithmic work."""
    d = w.d
    return {"attn": 12 * d * d, "ffn_head": flops_per_window(w)["ffn_head"]}


def measure_gated(wid, n, variants):
    """The gated loop of Alg. 1 with the controller of Alg. 2 (trace_gated_run:
    speculative forwards over up to 64 steps, exact by construction) over n
    steps of workload wid, for each (name, mode, delta) in variants, each from
    the workload's initial weights.  Per variant: bytes/s, updates (overall and
    after the warm-up), bits/byte (mean step cross-entropy), per-kind kernel
    times, Adam's bytes per launch against HBM; for the adaptation workload the
    update fraction and bits/byte in each 2 KiB source regime."""
    import numpy as np
    import torch
    import paper_2203_16114_amd as P
    import synth
    from synth.workloads import REGIME_BYTES_PER_STREAM
    w = synth.WORKLOADS[wid]
    B = w.B
    n = min(n, w.L - w.W)            # targets at positions W .. W + n - 1
    L = w.W + n
    t0 = time.time()
    streams, _ = synth.workload_streams(wid, L=L)
    log(f"[bench] {w.name} streams {streams.shape} in {time.time() - t0:.1f}s")
    sdev = torch.from_numpy(streams).cuda()
    mk = lambda: P.TraceModel(w.W, w.e, w.g, w.H, w.F, w.k, dtype=w.dtype, max_windows=B * 64, max_keep=B)
    warm = mk()                                  # first launches of every kernel, untimed
    warm.init_weights(w.weight_seed)
    warm.gated_run(sdev, w.W, 80, P.MODE_GATED, w.t, 0.0)
    warm.close()
    res = {"workload": f"{w.name}: B={B} windows/step, W={w.W} e={w.e} g={w.g} d={w.d} H={w.H} F={w.F} "
                       f"k={w.k}, controller t={w.t}; targets at positions {w.W}..{w.W + n - 1} of every stream",
           "steps": n}
    for name, mode, delta in variants:
        m = mk()
        m.init_weights(w.weight_seed)
        torch.cuda.synchronize()
        m.set_timing(True)
        t0 = time.perf_counter()
        ce, dec, upd = m.gated_run(sdev, w.W, n, mode, w.t, 0.0 if delta is None else delta)
        torch.cuda.synchronize()
        dt = time.perf_counter() - t0
        tm = m.read_timing()
        m.set_timing(False)
        r = {"mode": {P.MODE_GATED: "gated", P.MODE_ALWAYS: "always", P.MODE_NEVER: "never"}[mode],
             "delta_bits": delta, "bytes_per_s": B * n / dt, "seconds": round(dt, 3), "updates": upd,
             "update_fraction": round(upd / n, 5),
             "updates_after_warmup": int(dec[w.t:].sum()),
             "update_fraction_after_warmup": round(float(dec[w.t:].mean()), 5),
             "bits_per_byte": float(ce.mean()),
             "kernel_ms": {k: round(v[0], 3) for k, v in tm.items() if k != "overflow" and v[1]},
             "kernel_launches": {k: v[1] for k, v in tm.items() if k != "overflow" and v[1]}}
        if tm.get("backward", (0, 0))[1]:
            r["backward_ms_per_update"] = round(tm["backward"][0] / tm["backward"][1], 4)
        if tm.get("adam", (0, 0))[1]:
            ms = tm["adam"][0] / tm["adam"][1]
            # Adam moves 28 bytes per parameter: reads theta, g, m, v; writes theta, m, v
            r["adam"] = {"avg_launch_ms": round(ms, 5), "bytes_per_launch": 28 * m.n_params,
                         "hbm_frac": round((28.0 * m.n_params / (ms * 1e-3)) / (HBM_GBS * 1e9), 4)}
        if wid == 4:
            pos = w.W + np.arange(n)
            reg = pos // REGIME_BYTES_PER_STREAM
            r["per_regime"] = [{"regime": int(q), "steps": int((reg == q).sum()),
                                "update_fraction": round(float(dec[reg == q].mean()), 4),
                                "bits_per_byte": round(float(ce[reg == q].mean()), 5)}
                               for q in np.unique(reg)]
        res[name] = r
        log(f"[bench] {w.name} {name}: {r['bytes_per_s']:.4g} B/s, updates {upd}/{n}, "
            f"bits/byte {r['bits_per_byte']:.5f}")
        m.close()
    if "always_update" in res:
        base = res["always_update"]
        for name in res:
            if isinstance(res[name], dict) and name != "always_update" and "bytes_per_s" in res[name]:
                res[name]["speedup_vs_always"] = round(res[name]["bytes_per_s"] / base["bytes_per_s"], 4)
                res[name]["bits_per_byte_cost_vs_always"] = round(
                    (res[name]["bits_per_byte"] - base["bits_per_byte"]) / base["bits_per_byte"], 6)
    return res


def measure_forward(wid, steps_per_call, calls):
    """Forward estimator + code lengths on workload wid: `calls` launches of
    B x steps_per_call windows walking along the streams (one untimed first),
    timed with HIP events on the launch stream; per-kernel launch times and
    the fraction of the MFMA peak of the workload's dtype."""
    import torch
    import paper_2203_16114_amd as P
    import synth
    w = synth.WORKLOADS[wid]
    B, S = w.B, steps_per_call
    L = min(w.L, w.W + (calls + 1) * S + 1)
    streams, _ = synth.workload_streams(wid, L=L)
    sdev = torch.from_numpy(streams).cuda()
    m = P.TraceModel(w.W, w.e, w.g, w.H, w.F, w.k, dtype=w.dtype, max_windows=B * S)
    m.init_weights(w.weight_seed)
    bits = torch.empty(B * S, dtype=torch.float32, device="cuda")
    ce = torch.empty(calls, S, dtype=torch.float64, device="cuda")
    pos = [w.W + ((i + 1) * S) % max(L - w.W - S, 1) for i in range(calls)]
    m.forward_bits(sdev, w.W, S, bits=bits)
    torch.cuda.synchronize()
    m.set_timing(True)
    m.read_timing()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for i in range(calls):
        m.forward_bits(sdev, pos[i], S, bits=bits, step_ce=ce[i])
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1)
    tm = m.read_timing()
    m.set_timing(False)
    fpw = flops_per_window(w)
    wpl = B * S
    per = {k: tm[k][0] / max(tm[k][1], 1) for k in ("attn", "ffn_head")}
    peak = PEAK_TFLOPS[w.dtype]
    value = wpl * calls / (ms * 1e-3)
    path = (fpw["attn"] + fpw["ffn_head"]) * value / 1e12
    m.close()
    res = {"workload": f"{w.name}: B={B} streams x {S} positions per launch (first {L} bytes of each), "
                       f"W={w.W} e={w.e} g={w.g} d={w.d} H={w.H} F={w.F} k={w.k}, {w.dtype}",
           "bytes_per_s": value, "launches": calls, "windows_per_launch": wpl, "ms_per_launch": round(ms / calls, 4),
           "bits_per_byte": float(ce.mean()), "dtype": w.dtype, "peak_tflops": peak,
           "kernels": {k: {"avg_launch_ms": round(per[k], 4),
                           "tflops": round(fpw[k] * wpl / (per[k] * 1e-3) / 1e12, 2),
                           "frac": round(fpw[k] * wpl / (per[k] * 1e-3) / 1e12 / peak, 4)} for k in per},
           "path_tflops": round(path, 2), "path_frac": round(path / peak, 4)}
    log(f"[bench] forward {w.name}: {value:.4g} B/s, path {path:.1f} TFLOP/s ({path / peak:.3f} of {peak})")
    return res


def attn_kernel(w, steps_per_call):
    """The attention kernel of a forward launch: bf16 launches of whole
    64-window tiles per stream share the byte groups between windows, one
    head per wave at d = 256 with 8 heads and g = 8 (k_attn_wh), one window
    class per wave otherwise (k_attn_grp); the per-token kernel (k_attn) for
    the rest."""
    if w.dtype != "bf16" or steps_per_call % 64:
        return "k_attn"
    if w.d == 256 and w.H == 8 and w.g == 8 and w.T in (4, 8):
        return "k_attn_wh"
    return "k_attn_grp"


def traffic_for(kernel, windows_per_launch):
    """HBM bytes per launch of `kernel` from the committed counter summary
    (profiles/hbm_traffic.json: FETCH_SIZE and WRITE_SIZE per dispatch, scaled by
    the factors a 1 GiB device copy gives), or None when the summary is missing
    or was taken on a different version of the kernel's source."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "hbm_traffic.json")
    try:
        rec = json.load(open(path))["kernels"][kernel]
        src = os.path.join(ROOT, "paper_2203_16114_amd", "csrc", rec["source"])
        if hashlib.sha256(open(src, "rb").read()).hexdigest() != rec["source_sha256"]:
            return None
        per_window = rec["hbm_bytes_per_launch"] / rec["windows_per_launch"]
        return per_window * windows_per_launch
    except (OSError, KeyError, ValueError):
        return None


def cpu_baseline(streams, w, n_windows, n_windows_one_core):
    """The oracle, as it stands, on seeded windows of the main workload: on all
    of this machine's cores, then pinned to one core with one BLAS thread."""
    import numpy as np
    import oracle as O
    import synth
    try:
        from threadpoolctl import threadpool_info, threadpool_limits
        threads = max([x.get("num_threads", 1) for x in threadpool_info()] or [1])
    except Exception:
        threadpool_limits, threads = None, None
    cores = len(os.sched_getaffinity(0))
    cfg = O.Config(W=w.W, e=w.e, g=w.g, H=w.H, F=w.F, k=w.k)
    flat = O.init_flat(cfg, w.weight_seed)
    b, i = synth.sample_positions(0xBA5E, streams.shape[0], streams.shape[1], w.W, n_windows)
    win, y = O.windows_at(streams, b, i, w.W)
    mode = "bf16" if w.dtype == "bf16" else "fp64"
    O.forward(flat, cfg, win[:64], y[:64], mode=mode)       # first-call costs, untimed
    t0 = time.perf_counter()
    O.forward(flat, cfg, win, y, mode=mode)
    dt = time.perf_counter() - t0
    out = {"value": n_windows / dt, "unit": "bytes/s", "cores": threads or cores, "kind": "oracle",
           "sample": f"{n_windows} seeded windows of the {w.name} streams, oracle forward + code length in "
                     f"{mode} mode (numpy, {threads} BLAS threads on {cores} host cores), {dt:.1f} s"}
    if n_windows_one_core > 0 and threadpool_limits is not None:
        keep = os.sched_getaffinity(0)
        try:
            os.sched_setaffinity(0, {min(keep)})
            with threadpool_limits(1):
                nw = n_windows_one_core
                t0 = time.perf_counter()
                O.forward(flat, cfg, win[:nw], y[:nw], mode=mode)
                dt1 = time.perf_counter() - t0
        finally:
            os.sched_setaffinity(0, keep)
        out["one_core"] = {"value": nw / dt1, "unit": "bytes/s", "cores": 1,
                           "sample": f"the first {nw} of those windows, pinned to one core, one BLAS thread, "
                                     f"{dt1:.1f} s"}
    return out


def measure_codec(wid, n):
    """The compressor of Alg. 1 (trace_compress, then trace_decompress on a
    fresh model in the same starting state) over n positions past the window of
    every stream of workload wid, with the controller gating updates: real code
    bytes against the model's estimated bits, both directions timed, and the
    decoded streams compared with the input."""
    import torch
    import paper_2203_16114_amd as P
    import synth
    w = synth.WORKLOADS[wid]
    L = w.W + n
    streams, _ = synth.workload_streams(wid, L=L)
    sdev = torch.from_numpy(streams).cuda()
    mk = lambda: P.TraceModel(w.W, w.e, w.g, w.H, w.F, w.k, dtype=w.dtype, max_windows=w.B, max_keep=w.B)
    warm = mk()                                  # first launches and allocations, untimed
    warm.init_weights(w.weight_seed)
    warm.decompress(warm.compress(sdev[:8, :w.W + 4].contiguous())[0], w.W + 4)
    enc, dec = mk(), mk()
    enc.init_weights(w.weight_seed)
    dec.init_weights(w.weight_seed)
    torch.cuda.synchronize()
    t0 = time.time()
    codes, nu = enc.compress(sdev, mode=P.MODE_GATED, t=16, delta=0.05)
    t1 = time.time()
    out, nu2 = dec.decompress(codes, L, mode=P.MODE_GATED, t=16, delta=0.05)
    torch.cuda.synchronize()
    t2 = time.time()
    nbytes = w.B * L
    code_bytes = sum(len(c) for c in codes)
    res = {"workload": w.name, "streams": w.B, "bytes_per_stream": L, "updates": nu,
           "round_trip_exact": bool(torch.equal(out, sdev)) and nu == nu2,
           "code_bits_per_byte": round(8.0 * code_bytes / nbytes, 4),
           "compress_bytes_per_s": nbytes / (t1 - t0), "decompress_bytes_per_s": nbytes / (t2 - t1)}
    log(f"[bench] codec {w.name}: {res}")
    return res


def measure_sweep():
    """Synthetic analogues of the paper's Eq. 5 study (Fig. 3) and of its
    batch-size table: (1) for attention width d in {128, 256} and FFN width F in
    {512, ..., 4096} (W=32, g=4, T=8, k=2, bf16), the model adapts, updating at
    every step, on 512 streams (the paper's batch) drawn from ONE order-1 Markov
    source with Dirichlet(0.1) rows (context every stream shares, which a shared
    model can learn); after 1024 and after 4096 updates its compression ratio
    CR = 8 / (bits per byte of the next 64 positions, no update) and its latency
    t (one forward step over the 512 windows) give LCR = (t - t0) / (CR - CR0)
    against (d, F) = (128, 512); (2) forward throughput and the model's device
    memory of the main workload's model at 128 to 8192 streams of 256 positions."""
    import numpy as np
    import torch
    import paper_2203_16114_amd as P
    import synth
    B, S_ev = 512, 64
    checkpoints = (1024, 4096)
    S_ad = checkpoints[-1]
    streams, codelen = synth.shared_markov_streams(B, 32 + S_ad + S_ev + 1, 1, 0.1, 0x7ACE5EED)
    ideal = float(codelen.sum() / streams.size)
    sdev = torch.from_numpy(streams).cuda()
    rows = []
    for d in (128, 256):
        for F in (512, 1024, 2048, 4096):
            m = P.TraceModel(32, d // 4, 4, d // 32, F, 2, dtype="bf16", max_windows=B * S_ev, max_keep=B)
            m.init_weights(7)
            done = 0
            for cp in checkpoints:
                m.gated_run(sdev, 32 + done, cp - done, P.MODE_ALWAYS)
                done = cp
                ce = torch.empty(S_ev, dtype=torch.float64, device="cuda")
                bits = torch.empty(B * S_ev, dtype=torch.float32, device="cuda")
                m.forward_bits(sdev, 32 + done, S_ev, bits=bits, step_ce=ce)       # warm
                torch.cuda.synchronize()
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record()
                m.forward_bits(sdev, 32 + done, S_ev, bits=bits, step_ce=ce)
                e1.record()
                torch.cuda.synchronize()
                bpb = float(ce.mean())
                rows.append({"d": d, "F": F, "updates": cp, "bits_per_byte": round(bpb, 4),
                             "cr": round(8.0 / bpb, 4), "ms_per_step": round(e0.elapsed_time(e1) / S_ev, 4)})
                log(f"[bench] sweep {rows[-1]}")
            del m
    for cp in checkpoints:
        sel = [r for r in rows if r["updates"] == cp]
        r0 = sel[0]
        for r in sel[1:]:
            dcr = r["cr"] - r0["cr"]
            r["lcr_ms"] = round((r["ms_per_step"] - r0["ms_per_step"]) / dcr, 4) if abs(dcr) > 1e-6 else None
    w = synth.WORKLOADS[3]
    st, _ = synth.workload_streams(3, L=w.W + 256 * 4 + 1)
    st = np.concatenate([st, st[::-1]])[:8192]       # the workload holds 4096 streams
    batch = []
    for nb in (128, 512, 2048, 8192):
        sd = torch.from_numpy(np.ascontiguousarray(st[:nb])).cuda()
        torch.cuda.synchronize()
        free0 = torch.cuda.mem_get_info()[0]
        m = P.TraceModel(w.W, w.e, w.g, w.H, w.F, w.k, dtype=w.dtype, max_windows=nb * 256)
        m.init_weights(w.weight_seed)
        out = torch.empty(nb * 256, dtype=torch.float32, device="cuda")
        torch.cuda.synchronize()
        held = free0 - torch.cuda.mem_get_info()[0]
        m.forward_bits(sd, w.W, 256, bits=out)
        torch.cuda.synchronize()
        t0 = time.time()
        for i in range(3):
            m.forward_bits(sd, w.W + 256 * (i + 1), 256, bits=out)
        torch.cuda.synchronize()
        batch.append({"streams": nb, "bytes_per_s": round(nb * 256 * 3 / (time.time() - t0), 1),
                      "device_mib": round(held / 2**20, 1)})
        del m, out, sd
        log(f"[bench] batch {batch[-1]}")
    return {"lcr": rows, "lcr_source": "512 streams of one order-1 Markov source, Dirichlet(0.1) rows",
            "lcr_source_bits_per_byte": round(ideal, 4), "batch": batch}


def measure_performer(steps=3):
    """The Performer (FAVOR+) attention of the paper's experiments (Sec. 6)
    against exact softmax attention (Eqs. 1-2), forward + code lengths on the
    main workload's shape and streams, both models in the same process; the
    feature projection is seeded orthogonal random features."""
    import torch
    import paper_2203_16114_amd as P
    import synth
    w = synth.WORKLOADS[3]
    S = 256
    st, _ = synth.workload_streams(3, L=w.W + S * (steps + 1) + 1)
    sd = torch.from_numpy(st).cuda()
    B = st.shape[0]
    res = {"workload": w.name, "streams": B, "positions_per_step": S}
    for name, att in (("softmax", "softmax"), ("performer", "performer")):
        m = P.TraceModel(w.W, w.e, w.g, w.H, w.F, w.k, dtype=w.dtype, max_windows=B * S, attention=att)
        m.init_weights(w.weight_seed)
        if att == "performer":
            nf = 128 if w.d // w.H <= 32 else 256
            m.set_features(synth.performer_features(0x0FE43, nf, w.d // w.H))
            res["n_features"] = nf
        bits = torch.empty(B * S, dtype=torch.float32, device="cuda")
        m.forward_bits(sd, w.W, S, bits=bits)
        torch.cuda.synchronize()
        m.set_timing(True)
        m.read_timing()
        t0 = time.time()
        for i in range(steps):
            m.forward_bits(sd, w.W + S * (i + 1), S, bits=bits)
        torch.cuda.synchronize()
        res[name + "_bytes_per_s"] = B * S * steps / (time.time() - t0)
        tm = m.read_timing()
        res[name + "_attn_ms"] = round(tm["attn"][0] / max(tm["attn"][1], 1), 4)
        m.set_timing(False)
        del m
    res["performer_over_softmax"] = round(res["performer_bytes_per_s"] / res["softmax_bytes_per_s"], 4)
    log(f"[bench] performer {res}")
    return res


def measure_deep_ffn(steps=3):
    """The deep-FFN variant of Sec. 6.3 (untied W1, W2 per repeat) against the
    shared FFN on the main workload's shape and streams: forward bytes/s of
    4096 streams x 256 positions per step, both models in the same process."""
    import torch
    import paper_2203_16114_amd as P
    import synth
    w = synth.WORKLOADS[3]
    S = 256
    st, _ = synth.workload_streams(3, L=w.W + S * (steps + 1) + 1)
    sd = torch.from_numpy(st).cuda()
    B = st.shape[0]
    res = {"workload": w.name, "streams": B, "positions_per_step": S}
    for name, untied in (("shared", False), ("untied", True)):
        m = P.TraceModel(w.W, w.e, w.g, w.H, w.F, w.k, dtype=w.dtype, max_windows=B * S, untied_ffn=untied)
        m.init_weights(w.weight_seed)
        bits = torch.empty(B * S, dtype=torch.float32, device="cuda")
        m.forward_bits(sd, w.W, S, bits=bits)
        torch.cuda.synchronize()
        t0 = time.time()
        for i in range(steps):
            m.forward_bits(sd, w.W + S * (i + 1), S, bits=bits)
        torch.cuda.synchronize()
        res[name + "_bytes_per_s"] = B * S * steps / (time.time() - t0)
        res[name + "_params"] = m.n_params
        del m
    res["untied_over_shared"] = round(res["untied_bytes_per_s"] / res["shared_bytes_per_s"], 4)
    log(f"[bench] deep ffn {res}")
    return res


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=40)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--steps-per-call", type=int, default=256, help="positions per stream in one step")
    ap.add_argument("--full", action="store_true", help="generate the full 256 KiB streams")
    ap.add_argument("--adapt-steps", type=int, default=32736,
                    help="steps of each gated run on the adaptation workload (default: its whole streams; 0: skip)")
    ap.add_argument("--large-steps", type=int, default=4096,
                    help="steps of each gated run on the large mixed workload (0: skip)")
    ap.add_argument("--fwd-legs", type=int, default=1, help="forward legs of workloads 1, 2 and 5 (0: skip)")
    ap.add_argument("--cpu-windows", type=int, default=16384, help="oracle sample (0: skip)")
    ap.add_argument("--cpu-windows-one-core", type=int, default=1024, help="oracle sample on one core (0: skip)")
    ap.add_argument("--codec-steps", type=int, default=64, help="positions of the compress / decompress run (0: skip)")
    ap.add_argument("--sweep", action="store_true", help="only the LCR and batch-size sweeps (one JSON line)")
    ap.add_argument("--update-profile", type=int, default=0,
                    help="only run --update-steps always-update steps of this workload (4 or 5) "
                         "and print one JSON line: the run that the update's kernel profiles come from")
    ap.add_argument("--update-steps", type=int, default=30)
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="only run 5 device-to-device copies of this many MiB (calibrates the HBM "
                         "byte counters FETCH_SIZE / WRITE_SIZE against a copy of known size)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(--gpus must be 1)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    import paper_2203_16114_amd as P
    import synth

    if args.sweep:
        print(json.dumps({"sweep": measure_sweep()}), flush=True)
        return
    if args.update_profile:
        w = synth.WORKLOADS[args.update_profile]
        n = args.update_steps
        streams, _ = synth.workload_streams(args.update_profile, L=w.W + n + 9)
        sd = torch.from_numpy(streams).cuda()
        m = P.TraceModel(w.W, w.e, w.g, w.H, w.F, w.k, dtype=w.dtype, max_windows=w.B * 64, max_keep=w.B)
        m.init_weights(w.weight_seed)
        m.gated_run(sd, w.W, 8, P.MODE_ALWAYS)                      # first launches, untimed
        torch.cuda.synchronize()
        m.set_timing(True)
        m.read_timing()
        t0 = time.perf_counter()
        m.gated_run(sd, w.W + 8, n, P.MODE_ALWAYS)
        torch.cuda.synchronize()
        dt = time.perf_counter() - t0
        tm = m.read_timing()
        print(json.dumps({"update_profile": w.name, "steps": n, "ms_per_step": dt / n * 1e3,
                          "kernel_ms_per_launch": {k: round(v[0] / v[1], 4) for k, v in tm.items()
                                                   if k != "overflow" and v[1]}}), flush=True)
        return
    if args.copy_probe_mib > 0:
        n = args.copy_probe_mib << 20
        src = torch.empty(n, dtype=torch.uint8, device="cuda").fill_(1)
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes": n, "copies": 5}), flush=True)
        return

    w = synth.WORKLOADS[3]
    B, S, K = w.B, args.steps_per_call, args.steps
    need = w.W + (args.warmup + K) * S + 1
    if need > w.L:
        raise SystemExit(f"steps x steps-per-call exceed the stream length {w.L}")
    L = w.L if args.full else need
    t0 = time.time()
    streams, _ = synth.workload_streams(3, L=L)
    log(f"[bench] main workload streams {streams.shape} in {time.time() - t0:.1f}s")
    sdev = torch.from_numpy(streams).cuda()
    model = P.TraceModel(w.W, w.e, w.g, w.H, w.F, w.k, dtype=w.dtype, max_windows=B * S)
    model.init_weights(w.weight_seed)
    bits = torch.empty(B * S, dtype=torch.float32, device="cuda")
    ce = torch.empty(K + args.warmup, S, dtype=torch.float64, device="cuda")
    pos = w.W
    for i in range(args.warmup):
        model.forward_bits(sdev, pos, S, bits=bits, step_ce=ce[i])
        pos += S
    torch.cuda.synchronize()
    model.set_timing(True)
    model.read_timing()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    ev0.record()
    for i in range(K):
        model.forward_bits(sdev, pos, S, bits=bits, step_ce=ce[args.warmup + i])
        pos += S
    ev1.record()
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1)
    tm = model.read_timing()
    model.set_timing(False)
    windows = B * S * K
    value = windows / (ms * 1e-3)
    bpb = float(ce[args.warmup:].mean())
    log(f"[bench] main: {K} steps x {B * S} windows in {ms:.1f} ms -> {value:.4g} bytes/s; {tm}")

    fpw = flops_per_window(w)
    xpw = mfma_flops_per_window(w)
    per = {k: tm[k][0] / max(tm[k][1], 1) for k in ("attn", "ffn_head")}
    dom = max(per, key=lambda k: tm[k][0])
    wpl = B * S
    achieved = fpw[dom] * wpl / (per[dom] * 1e-3) / 1e12
    peak = PEAK_TFLOPS[w.dtype]
    total_tflops = (fpw["attn"] + fpw["ffn_head"]) * value / 1e12
    # the FFN + head kernel is k_ffn_pipe in bf16, k_ffn_head in fp32
    attn_k = attn_kernel(w, S)
    kname = ("k_ffn_pipe" if w.dtype == "bf16" else "k_ffn_head") if dom == "ffn_head" else attn_k
    traffic = traffic_for(kname, wpl)
    roofline = {"bound": "mfma", "kernel": kname,
                "achieved": round(achieved, 2), "peak": peak, "unit": "TFLOP/s", "frac": round(achieved / peak, 4),
                "traffic": None if traffic is None else round(traffic),
                "flops_per_window": fpw[dom], "windows_per_launch": wpl, "avg_launch_ms": round(per[dom], 4),
                "kernels": {k: {"avg_launch_ms": round(per[k], 4),
                                "tflops": round(fpw[k] * wpl / (per[k] * 1e-3) / 1e12, 2),
                                "mfma_tflops": round(xpw[k] * wpl / (per[k] * 1e-3) / 1e12, 2)} for k in per},
                "path_tflops": round(total_tflops, 2), "path_frac": round(total_tflops / peak, 4),
                "path_mfma_frac": round((xpw["attn"] + xpw["ffn_head"]) * value / 1e12 / peak, 4)}

    out = {"metric": "bytes/sec estimated (fwd+bits) and with gated adapt; MFMA util; bits/byte",
           "value": value, "unit": "bytes/s", "n_gpus": 1, "steps": K, "warmup": args.warmup,
           "ms_per_step": ms / K, "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
           "dtype": "bf16", "data": "synthetic",
           "config": {"workload": f"{w.name}: B={B} streams (order-3 Markov Dirichlet(0.02) / Zipf(1.2) / "
                                  f"uniform thirds), the first {L} bytes of each {w.L}-byte stream generated, "
                                  f"{K} timed launches of {S} consecutive positions per stream; W={w.W} e={w.e} "
                                  f"g={w.g} -> T={w.T} d={w.d}, H={w.H}, F={w.F} shared x{w.k}, bf16 operands "
                                  f"fp32 accumulate",
                      "windows_per_step": B * S, "steps_per_call": S, "stream_prefix_bytes": L},
           "bits_per_byte": bpb, "mfma_util": roofline["path_mfma_frac"], "roofline": roofline}
    if args.fwd_legs:
        out["forward_legs"] = {"tiny-fp32": measure_forward(1, 4080, 5), "small-fp32": measure_forward(2, 256, 8),
                               "large-mixed-bf16": measure_forward(5, 64, 8)}
    variants = [("gated", P.MODE_GATED, 0.05), ("gated_eq7", P.MODE_GATED, 0.0),
                ("always_update", P.MODE_ALWAYS, None)]
    out["gated_adapt"] = {}
    if args.adapt_steps > 0:
        out["gated_adapt"]["adapt-bf16"] = measure_gated(4, args.adapt_steps, variants)
    if args.large_steps > 0:
        out["gated_adapt"]["large-mixed-bf16"] = measure_gated(5, args.large_steps, variants)
    if args.codec_steps > 0:
        out["codec"] = measure_codec(4, args.codec_steps)
        out["deep_ffn"] = measure_deep_ffn()
        out["performer"] = measure_performer()
    if args.cpu_windows > 0:
        out["cpu_baseline"] = cpu_baseline(streams, w, args.cpu_windows, args.cpu_windows_one_core)
        log(f"[bench] cpu oracle: {out['cpu_baseline']['value']:.4g} bytes/s")
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
