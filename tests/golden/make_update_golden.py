#!/usr/bin/env python3
"""Writes the oracle's expected values for the update parity tests at the
adaptation and large workloads' shapes (tests/test_gpu_update_shapes.py):

  update_adapt.json  config-4 model (d = 128, F = 512, k = 2, bf16), B = 4096
  update_large.json  config-5 model (d = 512, F = 2048, k = 3, bf16), B = 8192

Each holds, for the seeded streams and weights of that workload (synth/, the
same inputs the GPU test builds): sketches (tests/sketch.py) of the gradient
of one step at the initial weights and of the parameter change of one Adam
step; and a teacher-forced run of the gated loop (Alg. 1 with Alg. 2) over a
fixed update schedule: the step cross-entropies, the oracle controller's own
decisions and thresholds, and a sketch of the final master weights.

Calls only the oracle (oracle/) and the input generator (synth/).  The oracle
takes minutes per step at these sizes, which is why its results are stored.
Usage: python tests/golden/make_update_golden.py [adapt|large ...]"""
from __future__ import annotations

import json
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)
sys.path.insert(0, os.path.dirname(HERE))

import oracle as O  # noqa: E402
import synth  # noqa: E402
from sketch import sketch  # noqa: E402

# workload id, streams, first target position, teacher-forced steps, controller t
CASES = {
    # 24 steps before the source switch at byte 2048 of every stream, 40 after
    "adapt": dict(wid=4, B=4096, pos0=2024, n_steps=64, t=16, delta=0.05),
    "large": dict(wid=5, B=8192, pos0=700, n_steps=6, t=4, delta=0.05),
}
SKETCH_SEED = 0x5EED5


def schedule(n_steps: int, t: int) -> list:
    """Updates at every warm-up step (as the controller makes them), then on a
    seeded ~30 % of the steps, with runs of skipped steps between updates."""
    rng = np.random.default_rng(0xD0)
    return [1] * min(t, n_steps) + [int(rng.random() < 0.3) for _ in range(max(n_steps - t, 0))]


def make(name: str) -> dict:
    c = CASES[name]
    w = synth.WORKLOADS[c["wid"]]
    cfg = O.Config(W=w.W, e=w.e, g=w.g, H=w.H, F=w.F, k=w.k)
    L = c["pos0"] + c["n_steps"] + 1
    streams, _ = synth.workload_streams(c["wid"], L=L, B=c["B"])
    flat = O.init_flat(cfg, w.weight_seed)
    B, pos0 = c["B"], c["pos0"]
    t0 = time.time()
    win, y = O.windows_at(streams, np.arange(B), np.full(B, pos0), cfg.W)
    _, g = O.forward_backward(flat, cfg, win, y, mode="bf16")
    gflat = O.flatten(g, cfg, np.float32)
    opt = O.Adam(flat.size, cfg)
    th1 = opt.step(flat, gflat)
    dth = O.unflatten(th1.astype(np.float64) - flat.astype(np.float64), cfg)
    print(f"[{name}] gradient and Adam step in {time.time() - t0:.0f} s", flush=True)
    forced = schedule(c["n_steps"], c["t"])
    t0 = time.time()
    _, ce, dec, own, th = O.run_gated(flat, cfg, streams, pos0, c["n_steps"], c["t"], c["delta"], mode="bf16",
                                      forced_decisions=forced)
    print(f"[{name}] {c['n_steps']} teacher-forced steps in {time.time() - t0:.0f} s", flush=True)
    ctl = O.Controller(c["t"], c["delta"])
    thr = []
    for e in ce:
        thr.append(ctl.threshold() if len(ctl.ring) == ctl.t else None)
        ctl.decide(e)
    names = [n for n, _ in O.param_layout(cfg)]
    gp = O.unflatten(gflat, cfg)
    thp = O.unflatten(th, cfg)
    return {
        "workload": w.name, "wid": c["wid"], "B": B, "pos0": pos0, "n_steps": c["n_steps"],
        "stream_len": L, "weight_seed": w.weight_seed, "sketch_seed": SKETCH_SEED,
        "t": c["t"], "delta": c["delta"], "mode": "bf16",
        "grad": {n: sketch(gp[n], SKETCH_SEED) for n in names},
        "dtheta1": {n: sketch(dth[n], SKETCH_SEED) for n in names},
        "teacher": {"forced": forced, "ce": [float(x) for x in ce], "own": [int(x) for x in own],
                    "threshold": thr},
        "theta_final": {n: sketch(thp[n], SKETCH_SEED) for n in names},
    }


def main():
    for name in sys.argv[1:] or list(CASES):
        out = make(name)
        path = os.path.join(HERE, f"update_{name}.json")
        with open(path, "w") as f:
            json.dump(out, f, separators=(",", ":"))
        print(f"wrote {path} ({os.path.getsize(path)} bytes)", flush=True)


if __name__ == "__main__":
    main()
