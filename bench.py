#!/usr/bin/env python3
"""Throughput of TRACE's batched next-byte estimator on one MI355X.

A step is one call of the forward estimator with code lengths over a batch of
windows of the main workload (4096 streams, W = 64 bytes, e = 32, g = 8 -> 8
tokens of d = 256, 8 heads, FFN 1024 shared x3, bf16 operands with fp32
accumulation): `--steps-per-call` consecutive positions of every stream, i.e.
4096 x S windows.  Successive steps walk along the streams.  The value is
predicted bytes (= windows) per second over the timed steps, with the streams
already in device memory.

Besides the headline line this run measures the controller-gated update loop
against the always-update loop on the adaptation workload (the small model in
bf16 with fp32 master weights, B = 4096 windows per step, sources switching
every 2 KiB per stream) and on the large mixed workload (d = 512, B = 8192),
and times the CPU oracle on a bounded sample of the main workload's windows on
this machine's cores.

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
    (bf16, 64-window tiles within one stream): the attention block projects each
    wave's 16 byte-group rows (15 distinct groups of its 8 windows) to K and V
    once, 16 * 4d^2 / 8 = 8d^2 per window, plus q and Wo (2d^2 each); the
    scores and weighted sums run on the vector ALUs.  The FFN executes its
    algorithmic work."""
    d = w.d
    return {"attn": 12 * d * d, "ffn_head": flops_per_window(w)["ffn_head"]}


def gated_loop(model, sdev, B, pos0, n_steps, t, delta, always, max_spec=64):
    """Alg. 1 with the controller of Alg. 2 over B streams.  Forward passes run
    speculatively over up to max_spec steps at unchanged weights; the controller
    walks their step cross-entropies and at the first step it flags, that step
    is re-run keeping its activations and updated; the walk resumes after it."""
    import torch
    import paper_2203_16114_amd as P
    ctl = P.Controller(t, delta)
    dev = sdev.device
    bits = torch.empty(B * max_spec, dtype=torch.float32, device=dev)
    ce = torch.empty(max_spec, dtype=torch.float64, device=dev)
    kb = torch.empty(B, dtype=torch.float32, device=dev)
    kce = torch.empty(1, dtype=torch.float64, device=dev)
    i, updates, spec, ce_sum = 0, 0, 1, 0.0
    ce_dev = []
    while i < n_steps:
        if always:
            model.forward_bits(sdev, pos0 + i, 1, bits=kb, step_ce=kce, keep=True)
            model.adapt_step()
            ce_dev.append(kce.clone())
            i += 1
            updates += 1
            continue
        S = min(spec, n_steps - i)
        model.forward_bits(sdev, pos0 + i, S, bits=bits, step_ce=ce)
        ces = ce[:S].cpu().numpy()
        j = None
        for s in range(S):
            if ctl.decide(float(ces[s])):
                j = s
                break
        used = S if j is None else j + 1
        ce_sum += float(ces[:used].sum())
        if j is not None:
            model.forward_bits(sdev, pos0 + i + j, 1, bits=kb, keep=True)
            model.adapt_step()
            updates += 1
            spec = 1
        else:
            spec = min(max_spec, spec * 2)
        i += used
    if ce_dev:
        ce_sum = float(torch.cat(ce_dev).sum())
    return updates, ce_sum / n_steps


def measure_gated(wid, n):
    """Gated (controller) vs always-update loop over n steps of workload wid."""
    import torch
    import paper_2203_16114_amd as P
    import synth
    w = synth.WORKLOADS[wid]
    B = w.B
    L = min(w.L, w.W + 1 + 2 * n + 2 * 64 + 64)
    t0 = time.time()
    streams, _ = synth.workload_streams(wid, L=L)
    log(f"[bench] {w.name} streams {streams.shape} in {time.time() - t0:.1f}s")
    sdev = torch.from_numpy(streams).cuda()
    res = {}
    for name, always in (("gated", False), ("always_update", True)):
        m = P.TraceModel(w.W, w.e, w.g, w.H, w.F, w.k, dtype=w.dtype, max_windows=B * 64, max_keep=B)
        m.init_weights(w.weight_seed)
        gated_loop(m, sdev, B, w.W, 8, w.t, w.delta, always)      # warm-up, then a fresh start
        m.init_weights(w.weight_seed)
        torch.cuda.synchronize()
        m.set_timing(True)
        t0 = time.perf_counter()
        upd, bpb = gated_loop(m, sdev, B, w.W + 8, n, w.t, w.delta, always)
        torch.cuda.synchronize()
        dt = time.perf_counter() - t0
        tm = m.read_timing()
        m.set_timing(False)
        res[name] = {"bytes_per_s": B * n / dt, "steps": n, "updates": upd, "update_fraction": upd / n,
                     "bits_per_byte": bpb,
                     "kernel_ms": {k: round(v[0], 3) for k, v in tm.items() if k != "overflow" and v[1]},
                     "kernel_launches": {k: v[1] for k, v in tm.items() if k != "overflow" and v[1]}}
        if tm.get("adam", (0, 0))[1]:
            ms = tm["adam"][0] / tm["adam"][1]
            # Adam moves 28 bytes per parameter: reads theta, g, m, v; writes theta, m, v
            res[name]["adam"] = {"avg_launch_ms": round(ms, 5), "bytes_per_launch": 28 * m.n_params,
                                 "hbm_frac": round((28.0 * m.n_params / (ms * 1e-3)) / (HBM_GBS * 1e9), 4)}
        log(f"[bench] {w.name} {name}: {res[name]['bytes_per_s']:.4g} B/s, updates {upd}/{n}")
        m.close()
    res["speedup_gated_vs_always"] = res["gated"]["bytes_per_s"] / res["always_update"]["bytes_per_s"]
    res["workload"] = f"{w.name}: B={B} windows/step, W={w.W} e={w.e} g={w.g} d={w.d} H={w.H} F={w.F} k={w.k}, " \
                      f"t={w.t} delta={w.delta}"
    return res


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


def cpu_baseline(streams, w, n_windows):
    import numpy as np
    import oracle as O
    import synth
    try:
        from threadpoolctl import threadpool_info
        threads = max([x.get("num_threads", 1) for x in threadpool_info()] or [1])
    except Exception:
        threads = None
    cores = len(os.sched_getaffinity(0))
    cfg = O.Config(W=w.W, e=w.e, g=w.g, H=w.H, F=w.F, k=w.k)
    flat = O.init_flat(cfg, w.weight_seed)
    b, i = synth.sample_positions(0xBA5E, streams.shape[0], streams.shape[1], w.W, n_windows)
    win, y = O.windows_at(streams, b, i, w.W)
    mode = "bf16" if w.dtype == "bf16" else "fp64"
    t0 = time.perf_counter()
    O.forward(flat, cfg, win, y, mode=mode)
    dt = time.perf_counter() - t0
    return {"value": n_windows / dt, "unit": "bytes/s", "cores": threads or cores, "kind": "oracle",
            "sample": f"{n_windows} seeded windows of the {w.name} streams, oracle forward + code length in "
                      f"{mode} mode (numpy, {threads} BLAS threads on {cores} host cores), {dt:.1f} s"}


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
    {512, ..., 4096} (W=32, g=4, T=8, k=2, bf16), the model adapts on the small
    workload's stream mix (order-2 Markov and Zipf bytes), 512 streams (the
    paper's batch), with an update every step for 4096 steps; then its
    compression ratio CR = 8 / (bits per byte of the next 64 positions, no
    update) and its latency t (one forward step over the 512 windows) give
    LCR = (t - t0) / (CR - CR0) against (d, F) = (128, 512); (2) forward
    throughput and the model's device memory of the main workload's model at
    128 to 8192 streams of 256 positions."""
    import numpy as np
    import torch
    import paper_2203_16114_amd as P
    import synth
    B, S_ad, S_ev = 512, 4096, 64
    streams, _ = synth.workload_streams(2, L=32 + S_ad + S_ev + 1, B=B)
    assert streams.shape[0] == B
    sdev = torch.from_numpy(streams).cuda()
    rows = []
    for d in (128, 256):
        for F in (512, 1024, 2048, 4096):
            m = P.TraceModel(32, d // 4, 4, d // 32, F, 2, dtype="bf16", max_windows=B * S_ev, max_keep=B)
            m.init_weights(7)
            for i in range(S_ad):
                m.forward_bits(sdev, 32 + i, 1, keep=True)
                m.adapt_step()
            ce = torch.empty(S_ev, dtype=torch.float64, device="cuda")
            bits = torch.empty(B * S_ev, dtype=torch.float32, device="cuda")
            m.forward_bits(sdev, 32 + S_ad, S_ev, bits=bits, step_ce=ce)       # warm
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            m.forward_bits(sdev, 32 + S_ad, S_ev, bits=bits, step_ce=ce)
            e1.record()
            torch.cuda.synchronize()
            bpb = float(ce.mean())
            rows.append({"d": d, "F": F, "bits_per_byte": round(bpb, 4), "cr": round(8.0 / bpb, 4),
                         "ms_per_step": round(e0.elapsed_time(e1) / S_ev, 4)})
            del m
            log(f"[bench] sweep {rows[-1]}")
    r0 = rows[0]
    for r in rows[1:]:
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
    return {"lcr": rows, "batch": batch}


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
    ap.add_argument("--gated-steps", type=int, default=256, help="steps of each gated-adaptation run (0: skip)")
    ap.add_argument("--cpu-windows", type=int, default=16384, help="oracle sample (0: skip)")
    ap.add_argument("--codec-steps", type=int, default=64, help="positions of the compress / decompress run (0: skip)")
    ap.add_argument("--sweep", action="store_true", help="only the LCR and batch-size sweeps (one JSON line)")
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
    # bf16 launches of whole 64-window tiles per stream take the shared-group attention kernel
    attn_k = "k_attn_grp" if (w.dtype == "bf16" and S % 64 == 0) else "k_attn"
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
           "config": {"workload": f"{w.name}: B={B} streams x {w.L} bytes (order-3 Markov Dirichlet(0.02) / "
                                  f"Zipf(1.2) / uniform thirds), W={w.W} e={w.e} g={w.g} -> T={w.T} d={w.d}, "
                                  f"H={w.H}, F={w.F} shared x{w.k}, bf16 operands fp32 accumulate",
                      "windows_per_step": B * S, "steps_per_call": S, "stream_prefix_bytes": L},
           "bits_per_byte": bpb, "mfma_util": roofline["path_mfma_frac"], "roofline": roofline}
    if args.gated_steps > 0:
        out["gated_adapt"] = {"adapt-bf16": measure_gated(4, args.gated_steps),
                              "large-mixed-bf16": measure_gated(5, max(16, args.gated_steps // 2))}
    if args.codec_steps > 0:
        out["codec"] = measure_codec(4, args.codec_steps)
        out["deep_ffn"] = measure_deep_ffn()
    if args.cpu_windows > 0:
        out["cpu_baseline"] = cpu_baseline(streams, w, args.cpu_windows)
        log(f"[bench] cpu oracle: {out['cpu_baseline']['value']:.4g} bytes/s")
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
