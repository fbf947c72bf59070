"""Seeded generators for input spike trains, weights, delays and labels.

Every random draw is keyed by (seed, sample) or (seed, projection) through
NumPy's PCG64 SeedSequence, so sample b of a batch of 256 equals sample b of a
batch of 16.  Seeds: data 1000*c + 1, weights 1000*c + 2, labels 1000*c + 3 for
config c.  The shapes and rates stand in for the paper's datasets (SHD/SSC
audio spike trains, Braille tactile sequences, Yin-Yang latency codes, the
sequence-detection toy); no dataset item is reproduced.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import List, Optional, Sequence

import numpy as np

from .configs import CONFIGS, Config, projections, weight_means, weight_stds


def _rng(*key: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence(list(key)))


def _sample_bernoulli(rng, T, n_in, p_step):
    """p_step: scalar or [T][n_in] firing probability per (step, channel)."""
    u = rng.random((T, n_in))
    s, c = np.nonzero(u < p_step)
    return s, c


def _one_sample(cfg: Config, T: int, dt: float, n_in: int, rng: np.random.Generator):
    g, gp = cfg.generator, cfg.gen_params
    if g == "bernoulli":
        return _sample_bernoulli(rng, T, n_in, gp["rate_hz"] * dt * 1e-3)
    if g == "latency":
        t = rng.uniform(0.0, gp["t_max_ms"], size=n_in)
        steps = np.floor(t / dt).astype(np.int64)
        keep = steps < T
        return steps[keep], np.arange(n_in)[keep]
    if g == "bumps":
        tt = (np.arange(T) * dt)[:, None]
        rate = np.zeros((T, n_in))
        for _ in range(gp["n_bumps"]):
            mu = rng.uniform(0.0, T * dt, size=n_in)
            sd = rng.uniform(10.0, 50.0, size=n_in)
            wt = rng.uniform(0.5, 1.0, size=n_in)
            rate += wt * np.exp(-0.5 * ((tt - mu) / sd) ** 2)
        rate *= gp["peak_hz"] / rate.max(axis=0, keepdims=True)
        return _sample_bernoulli(rng, T, n_in, rate * dt * 1e-3)
    if g == "audio":
        n_spk = rng.poisson(gp["mean_spikes"])
        k = int(rng.integers(3, 7))
        centres = rng.uniform(0.0, n_in, size=k)
        widths = rng.uniform(15.0, 80.0, size=k)
        mix = rng.dirichlet(np.ones(k))
        ch = np.arange(n_in)[:, None]
        env = (mix * np.exp(-0.5 * ((ch - centres) / widths) ** 2) / widths).sum(axis=1)
        pmf = 0.95 * env / env.sum() + 0.05 / n_in
        pmf /= pmf.sum()
        chans = rng.choice(n_in, size=n_spk, p=pmf)
        t_on = rng.uniform(0.0, 200.0)
        t_off = min(t_on + rng.uniform(300.0, 800.0), T * dt)
        t = rng.uniform(t_on, t_off, size=n_spk)
        steps = np.floor(t / dt).astype(np.int64)
        keep = steps < T
        return steps[keep], chans[keep]
    raise ValueError(f"unknown generator {g}")


def input_spikes(cfg: Config, B: int, seed: Optional[int] = None, T: Optional[int] = None):
    """CSR over samples: offsets [B+1], step [nnz], neuron [nnz] (int32).
    Within a sample the events are sorted by (step, neuron) and unique."""
    seed = 1000 * cfg.cid + 1 if seed is None else seed
    T = cfg.T if T is None else T
    n_in = cfg.layers[0][0]
    offs = [0]
    steps, neurons = [], []
    for b in range(B):
        s, c = _one_sample(cfg, T, cfg.dt, n_in, _rng(seed, b))
        key = np.unique(s.astype(np.int64) * n_in + c.astype(np.int64))
        steps.append((key // n_in).astype(np.int32))
        neurons.append((key % n_in).astype(np.int32))
        offs.append(offs[-1] + key.size)
    return (np.asarray(offs, dtype=np.int32),
            np.concatenate(steps) if steps else np.zeros(0, np.int32),
            np.concatenate(neurons) if neurons else np.zeros(0, np.int32))


def weights_and_delays(cfg: Config, seed: Optional[int] = None,
                       mus: Optional[Sequence[float]] = None):
    """Per projection: W [n_pre][n_post] ~ N(mu_p, std_p) and
    D [n_pre][n_post] ~ U[0, range_p] in steps (fp32, unrounded)."""
    seed = 1000 * cfg.cid + 2 if seed is None else seed
    mus = weight_means(cfg) if mus is None else list(mus)
    sds = weight_stds(cfg)
    Ws, Ds = [], []
    for p, (a, q) in enumerate(projections(cfg.layers)):
        n_pre, n_post = cfg.layers[a][0], cfg.layers[q][0]
        rng = _rng(seed, p)
        W = rng.normal(mus[p], sds[p], size=(n_pre, n_post)).astype(np.float32)
        D = rng.uniform(0.0, float(cfg.delay_range[p]), size=(n_pre, n_post)).astype(np.float32)
        Ws.append(W)
        Ds.append(D)
    return Ws, Ds


def labels(cfg: Config, B: int, seed: Optional[int] = None):
    seed = 1000 * cfg.cid + 3 if seed is None else seed
    C = cfg.n_classes
    return np.asarray([int(_rng(seed, b).integers(C)) for b in range(B)], dtype=np.int32)


@dataclass
class Workload:
    cfg: Config
    B: int
    T: int
    in_off: np.ndarray
    in_step: np.ndarray
    in_neuron: np.ndarray
    W: List[np.ndarray]
    D: List[np.ndarray]
    labels: np.ndarray

    @property
    def layers(self):
        return self.cfg.layers


def make_workload(cid: int, B: Optional[int] = None, T: Optional[int] = None,
                  mus: Optional[Sequence[float]] = None, weight_scale: float = 1.0) -> Workload:
    cfg = CONFIGS[cid]
    B = cfg.B if B is None else B
    T = cfg.T if T is None else T
    off, st, ne = input_spikes(cfg, B, T=T)
    W, D = weights_and_delays(cfg, mus=mus)
    if weight_scale != 1.0:
        W = [(w * np.float32(weight_scale)).astype(np.float32) for w in W]
    return Workload(cfg, B, T, off, st, ne, W, D, labels(cfg, B))


def make_variant(cid: int, B: Optional[int] = None, T: Optional[int] = None,
                 dt: Optional[float] = None, delay_range: Optional[Sequence[int]] = None,
                 name: Optional[str] = None, layers=None, loss: Optional[int] = None,
                 dmse_delta: Optional[float] = None) -> Workload:
    """Config `cid` with another grid (dt, T), other delay ranges (in steps),
    or another output layer and loss (same layer sizes: a LIF output layer
    with the spike-time loss), drawn from the same seeds and weight means;
    the input generator keeps its rates and times in ms, so a finer dt
    resolves the same spike trains."""
    import dataclasses
    base = CONFIGS[cid]
    kw = {}
    if dt is not None:
        kw["dt"] = float(dt)
    if T is not None:
        kw["T"] = int(T)
    if delay_range is not None:
        if len(delay_range) != len(base.delay_range):
            raise ValueError("one delay range per projection")
        kw["delay_range"] = tuple(int(x) for x in delay_range)
    if layers is not None:
        if [l[0] for l in layers] != [l[0] for l in base.layers]:
            raise ValueError("a variant keeps the layer sizes")
        kw["layers"] = tuple(tuple(int(x) for x in l) for l in layers)
    if loss is not None:
        kw["loss"] = int(loss)
    if dmse_delta is not None:
        kw["dmse_delta"] = float(dmse_delta)
    cfg = dataclasses.replace(base, name=name or base.name, **kw)
    B = cfg.B if B is None else B
    off, st, ne = input_spikes(cfg, B, T=cfg.T)
    W, D = weights_and_delays(cfg, mus=weight_means(base))
    return Workload(cfg, B, cfg.T, off, st, ne, W, D, labels(cfg, B))
