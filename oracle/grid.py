"""ctypes driver for the C grid oracle (test infrastructure only)."""
from __future__ import annotations

import ctypes as C
import os
from dataclasses import dataclass
from typing import List, Optional, Sequence

import numpy as np

from . import build as _build

_lib = None


def lib_path() -> str:
    return _build.OUT


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_build.OUT):
            _build.build()
        lib = C.CDLL(_build.OUT)
        ip, fp, dp, lp = (C.POINTER(C.c_int), C.POINTER(C.c_float), C.POINTER(C.c_double),
                          C.POINTER(C.c_long))
        lib.oracle_constants.argtypes = [C.c_float, C.c_float, C.c_float, fp]
        lib.oracle_forward.argtypes = (
            [C.c_int, ip, ip, ip, C.c_float, C.c_float, C.c_float, C.c_float, C.c_int, ip,
             C.c_int, C.c_int, C.c_int, C.c_float, ip, ip, ip, fp, fp, C.c_int,
             ip, ip, ip, fp, fp, ip, fp, fp, fp, lp])
        lib.oracle_loss.argtypes = [C.c_int, C.c_int, fp, ip, fp, fp]
        lib.oracle_loss_dmse.argtypes = [C.c_int, C.c_int, fp, ip, C.c_float, fp, dp]
        lib.oracle_backward.argtypes = (
            [C.c_int, ip, ip, ip, C.c_float, C.c_float, C.c_float, C.c_float, C.c_int, ip,
             C.c_int, C.c_int, C.c_int, C.c_float, ip, ip, ip, fp, fp, C.c_int,
             ip, ip, ip, fp, fp, ip, dp, C.c_int, dp, dp, lp])
        for f in (lib.oracle_constants, lib.oracle_forward, lib.oracle_loss, lib.oracle_loss_dmse,
                  lib.oracle_backward):
            f.restype = C.c_int
        _lib = lib
    return _lib


def _p(a: Optional[np.ndarray], ctype):
    if a is None:
        return C.cast(0, C.POINTER(ctype))
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data_as(C.POINTER(ctype))


def _i32(a):
    return np.ascontiguousarray(a, dtype=np.int32)


def _f32(a):
    return np.ascontiguousarray(a, dtype=np.float32)


def constants(tau_m: float, tau_s: float, dt: float) -> np.ndarray:
    """(alpha, beta, gamma, c) as fp32, from fp64 host arithmetic."""
    out = np.zeros(4, np.float32)
    rc = _load().oracle_constants(tau_m, tau_s, dt, _p(out, C.c_float))
    if rc:
        raise ValueError(f"oracle_constants rc={rc}")
    return out


@dataclass
class OracleNet:
    layers: Sequence[Sequence[int]]     # (n, kind, recurrent)
    tau_m: float
    tau_s: float
    theta: float
    dt: float
    max_delay: int
    T: int
    loss: int
    readout_scale: float
    proj_max_delay: Optional[Sequence[int]] = None   # largest delay per projection (None: max_delay)

    @property
    def L(self):
        return len(self.layers)

    def arrays(self):
        n = _i32([l[0] for l in self.layers])
        k = _i32([l[1] for l in self.layers])
        r = _i32([l[2] for l in self.layers])
        return n, k, r

    def pmax(self):
        return None if self.proj_max_delay is None else _i32(self.proj_max_delay)

    @property
    def n_lif(self):
        return sum(1 for l in self.layers if l[1] == 1)

    @property
    def cap_layers(self):
        """Layers whose spikes are recorded (every LIF layer, output included)."""
        return [l for l in self.layers[1:] if l[1] == 1]

    @property
    def n_state(self):
        return sum(l[0] for l in self.layers[1:])


@dataclass
class ForwardResult:
    rc: int
    count: np.ndarray       # [n_lif][B]
    step: np.ndarray        # [n_lif][B][cap]
    neuron: np.ndarray
    I_minus: np.ndarray
    z: np.ndarray           # [B][C]
    nstar: np.ndarray       # [B][C]
    V_final: np.ndarray     # [B][n_state]
    I_final: np.ndarray
    V_trace: Optional[np.ndarray]
    clamped: int
    cap: int

    def spikes(self, li: int, b: int):
        c = min(int(self.count[li, b]), self.cap)
        return self.step[li, b, :c], self.neuron[li, b, :c]


def _flat(arrs: Sequence[np.ndarray]) -> np.ndarray:
    return _f32(np.concatenate([np.ravel(np.asarray(a, dtype=np.float32)) for a in arrs]))


def forward(net: OracleNet, in_off, in_step, in_neuron, W: Sequence[np.ndarray],
            D: Sequence[np.ndarray], cap: Optional[int] = None, trace: bool = False) -> ForwardResult:
    lib = _load()
    n, k, r = net.arrays()
    in_off, in_step, in_neuron = _i32(in_off), _i32(in_step), _i32(in_neuron)
    B = in_off.size - 1
    C_ = net.layers[-1][0]
    if cap is None:
        cap = net.T * max([l[0] for l in net.cap_layers] + [1])
    nl = max(net.n_lif, 1)
    cnt = np.zeros((nl, B), np.int32)
    st = np.zeros((nl, B, cap), np.int32)
    ne = np.zeros((nl, B, cap), np.int32)
    Im = np.zeros((nl, B, cap), np.float32)
    z = np.zeros((B, C_), np.float32)
    ns = np.zeros((B, C_), np.int32)
    Vf = np.zeros((B, net.n_state), np.float32)
    If = np.zeros((B, net.n_state), np.float32)
    Vt = np.zeros((B, net.T, net.n_state), np.float32) if trace else None
    stats = np.zeros(4, np.int64)
    Wf, Df = _flat(W), _flat(D)
    pm = net.pmax()
    rc = lib.oracle_forward(net.L, _p(n, C.c_int), _p(k, C.c_int), _p(r, C.c_int),
                            net.tau_m, net.tau_s, net.theta, net.dt, net.max_delay, _p(pm, C.c_int),
                            B, net.T, net.loss, net.readout_scale,
                            _p(in_off, C.c_int), _p(in_step, C.c_int), _p(in_neuron, C.c_int),
                            _p(Wf, C.c_float), _p(Df, C.c_float), cap,
                            _p(cnt, C.c_int), _p(st, C.c_int), _p(ne, C.c_int), _p(Im, C.c_float),
                            _p(z, C.c_float), _p(ns, C.c_int), _p(Vf, C.c_float), _p(If, C.c_float),
                            _p(Vt, C.c_float), _p(stats, C.c_long))
    if rc not in (0, -4):
        raise ValueError(f"oracle_forward rc={rc}")
    return ForwardResult(rc, cnt, st, ne, Im, z, ns, Vf, If, Vt, int(stats[0]), cap)


def loss(z: np.ndarray, labels) -> tuple:
    z = _f32(z)
    labels = _i32(labels)
    B, C_ = z.shape
    lo = np.zeros(B + 1, np.float32)
    g = np.zeros((B, C_), np.float32)
    rc = _load().oracle_loss(B, C_, _p(z, C.c_float), _p(labels, C.c_int), _p(lo, C.c_float),
                             _p(g, C.c_float))
    if rc:
        raise ValueError(f"oracle_loss rc={rc}")
    return lo, g


LOSS_DMSE = 2


def loss_dmse(z: np.ndarray, labels, delta: float) -> tuple:
    """Time-invariant MSE on first output spike times z [B][C] (ms): per-sample
    and mean loss [B+1] (fp32) and dL/dt_k of the batch mean [B][C] (fp64)."""
    z = _f32(z)
    labels = _i32(labels)
    B, C_ = z.shape
    lo = np.zeros(B + 1, np.float32)
    dl = np.zeros((B, C_), np.float64)
    rc = _load().oracle_loss_dmse(B, C_, _p(z, C.c_float), _p(labels, C.c_int), float(delta),
                                  _p(lo, C.c_float), _p(dl, C.c_double))
    if rc:
        raise ValueError(f"oracle_loss_dmse rc={rc}")
    return lo, dl


def first_spike_dlp(net: OracleNet, fwd: ForwardResult, dl: np.ndarray) -> np.ndarray:
    """Per-record dl_p/dt_k [n_lif][B][cap] for the time-invariant MSE: the
    first spike of output neuron k in sample b carries dl[b][k], every other
    record 0 (later spikes do not enter the loss)."""
    nl = max(net.n_lif, 1)
    B, cap = fwd.count.shape[1], fwd.cap
    out = np.zeros((nl, B, cap), np.float64)
    li = net.n_lif - 1                       # the output layer is the last LIF layer
    for b in range(B):
        seen = set()
        for r in range(min(int(fwd.count[li, b]), cap)):
            k = int(fwd.neuron[li, b, r])
            if k not in seen:
                seen.add(k)
                out[li, b, r] = dl[b, k]
    return out


def spike_count_reg(net: OracleNet, fwd: ForwardResult, strength: Sequence[float],
                    target: float):
    """Hidden spike-count regulariser (Results, SHD/SSC/Braille: a target
    number of spikes per example and a layer-wise strength), read as: with
    cbar_i the batch-mean spike count of neuron i of LIF layer l, the penalty
    R = sum_l strength_l / 2 sum_i (cbar_i - target)^2, and every recorded
    spike of neuron i carries dl_p/dt_k = -strength_l (cbar_i - target) / B
    into its jump.  Returns (R, dlp [n_lif][B][cap] fp64)."""
    nl = max(net.n_lif, 1)
    B, cap = fwd.count.shape[1], fwd.cap
    sizes = [l[0] for l in net.layers if l[1] == 1]
    dlp = np.zeros((nl, B, cap), np.float64)
    R = 0.0
    for li, n in enumerate(sizes):
        rho = float(strength[li])
        if rho == 0.0:
            continue
        counts = np.zeros(n, np.int64)
        for b in range(B):
            c = min(int(fwd.count[li, b]), cap)
            np.add.at(counts, fwd.neuron[li, b, :c], 1)
        cbar = counts / float(B)
        R += 0.5 * rho * float(np.sum((cbar - target) ** 2))
        term = -rho * (cbar - target) / float(B)
        for b in range(B):
            c = min(int(fwd.count[li, b]), cap)
            dlp[li, b, :c] = term[fwd.neuron[li, b, :c]]
    return R, dlp


def backward(net: OracleNet, in_off, in_step, in_neuron, W: Sequence[np.ndarray],
             D: Sequence[np.ndarray], fwd: ForwardResult, g: np.ndarray, mode: str = "f64",
             dlp: Optional[np.ndarray] = None):
    """Returns (dW list, dD list, degenerate count); fp64 arrays shaped like W.
    g: dL/dz of the voltage readout (CE losses; ignored for the spike-time
    loss).  dlp: per-record dl_p/dt_k [n_lif][B][cap] (fp64) added to the
    jump of every recorded spike, or None."""
    lib = _load()
    n, k, r = net.arrays()
    in_off, in_step, in_neuron = _i32(in_off), _i32(in_step), _i32(in_neuron)
    B = in_off.size - 1
    Wf, Df = _flat(W), _flat(D)
    dW = np.zeros(Wf.size, np.float64)
    dD = np.zeros(Wf.size, np.float64)
    stats = np.zeros(4, np.int64)
    g = _f32(g)
    if dlp is not None:
        dlp = np.ascontiguousarray(dlp, dtype=np.float64)
        assert dlp.shape == (max(net.n_lif, 1), B, fwd.cap)
    pm = net.pmax()
    rc = lib.oracle_backward(net.L, _p(n, C.c_int), _p(k, C.c_int), _p(r, C.c_int),
                             net.tau_m, net.tau_s, net.theta, net.dt, net.max_delay, _p(pm, C.c_int),
                             B, net.T, net.loss, net.readout_scale,
                             _p(in_off, C.c_int), _p(in_step, C.c_int), _p(in_neuron, C.c_int),
                             _p(Wf, C.c_float), _p(Df, C.c_float), fwd.cap,
                             _p(fwd.count, C.c_int), _p(fwd.step, C.c_int), _p(fwd.neuron, C.c_int),
                             _p(fwd.I_minus, C.c_float), _p(g, C.c_float), _p(fwd.nstar, C.c_int),
                             _p(dlp, C.c_double), {"f64": 0, "f32": 1}[mode],
                             _p(dW, C.c_double), _p(dD, C.c_double), _p(stats, C.c_long))
    if rc:
        raise ValueError(f"oracle_backward rc={rc}")
    outW, outD, o = [], [], 0
    for w in W:
        sz = np.asarray(w).size
        outW.append(dW[o:o + sz].reshape(np.asarray(w).shape))
        outD.append(dD[o:o + sz].reshape(np.asarray(w).shape))
        o += sz
    return outW, outD, int(stats[0])
