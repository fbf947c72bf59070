"""Calibrate the feed-forward weight means into LIF layers (test infrastructure).

For each configuration with a target activity, and each feed-forward projection
into a LIF layer in projection order, bisect the weight mean mu so that the
oracle forward over the first samples of the batch (the whole batch, at most 32
samples for the two-layer 1024-neuron config whose oracle is slow) gives the
target mean number of spikes per neuron per sample in that projection's post
layer (about 14, the hidden
spike-count target the paper uses on SHD; about 1 for the latency-coded
config).  Writes ``workloads/calibration.json``; run once:

    python -m oracle.calibrate [config ids]
"""
from __future__ import annotations

import json
import os
import sys

import numpy as np

from workloads import CONFIGS, projections
from workloads.configs import _CAL_PATH
from workloads.generators import input_spikes, weights_and_delays

from . import grid

MAX_SAMPLES_WIDE = 32       # for networks wider than 512 LIF neurons


def n_samples(cfg):
    wide = sum(n for n, k, _ in cfg.layers if k == 1) > 512
    return min(cfg.B, MAX_SAMPLES_WIDE) if wide else cfg.B


def _rate(cfg, mus, layer, off, st, ne):
    W, D = weights_and_delays(cfg, mus=mus)
    net = grid.OracleNet(cfg.layers, cfg.tau_m, cfg.tau_s, cfg.theta, cfg.dt, cfg.max_delay, cfg.T,
                         cfg.loss, cfg.readout_scale)
    f = grid.forward(net, off, st, ne, W, D)
    li = [l for l in range(len(cfg.layers)) if cfg.layers[l][1] == 1].index(layer)
    return f.count[li].sum() / ((len(off) - 1) * cfg.layers[layer][0])


def calibrate(cid: int):
    cfg = CONFIGS[cid]
    mus = [m for m, _ in cfg.w_init]
    if cfg.target_rate <= 0:
        return mus
    off, st, ne = input_spikes(cfg, n_samples(cfg))
    for p, (a, q) in enumerate(projections(cfg.layers)):
        if p not in cfg.calibrate:
            continue
        lo, hi = 0.0, 0.05
        while True:
            mus[p] = hi
            r = _rate(cfg, mus, q, off, st, ne)
            print(f"cfg{cid} p{p} mu={hi:.6g} rate={r:.3f}", flush=True)
            if r >= cfg.target_rate:
                break
            lo, hi = hi, hi * 2.0
        for _ in range(30):
            mid = 0.5 * (lo + hi)
            mus[p] = mid
            r = _rate(cfg, mus, q, off, st, ne)
            if r < cfg.target_rate:
                lo = mid
            else:
                hi = mid
            if hi - lo < 1e-5 * hi:
                break
        mus[p] = hi
        print(f"cfg{cid} p{p} -> mu={hi:.6g} rate={_rate(cfg, mus, q, off, st, ne):.3f}", flush=True)
    return mus


def main(argv):
    ids = [int(a) for a in argv] if argv else sorted(CONFIGS)
    try:
        with open(_CAL_PATH) as f:
            cal = json.load(f)
    except FileNotFoundError:
        cal = {}
    for cid in ids:
        mus = calibrate(cid)
        cal[str(cid)] = {"mu": {str(p): float(mus[p]) for p in CONFIGS[cid].calibrate},
                         "target_spikes_per_neuron": CONFIGS[cid].target_rate,
                         "samples": n_samples(CONFIGS[cid])}
        with open(_CAL_PATH, "w") as f:
            json.dump(cal, f, indent=1, sort_keys=True)
    return 0


if __name__ == "__main__":
    sys.exit(main(sys.argv[1:]))
