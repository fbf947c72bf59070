"""Exact continuous-time simulator and EventProp backward for tiny networks.

TEST INFRASTRUCTURE ONLY (fp64, pure Python, a handful of neurons).  It pins
the grid oracle: its gradients are checked against central finite differences
of the exact loss, and the grid oracle is checked to converge to them as the
time step shrinks.

Model (Table 1): tau_m V' = -V + I, tau_s I' = -I between events; a LIF neuron
spikes when V reaches theta from below and is reset to 0; a spike of neuron n
at t_k makes I_m jump by w_mn at t_k + d_mn (real-valued delays >= 0).  The
readout layer is LI (no threshold), or LIF for the spike-time loss.  Loss,
with per-readout weights c_k:
  "integral":  L = sum_k c_k * integral_0^T V_k dt   (a voltage loss l_V)
  "max":       L = sum_k c_k * max_t V_k(t)          (source at t_max)
  "dmse":      L = 1/2 sum_{i != c} (t_i - t_c - Delta)^2 on the first spike
               times t_i of a LIF output layer (T if none; c the label), the
               time-invariant MSE of the Methods (a spike-time loss l_p)
and optionally a spike-time term coef_l * t_k for every spike of a chosen
LIF layer l (lp_lin = {l: coef_l}), and the spike-count regulariser
(spike_reg = {l: (rho, nu)}) read on one sample: with c_i the spike count of
neuron i of layer l in this run, the term -rho (c_i - nu) t_k for every spike
k of neuron i (c_i is constant under the small parameter steps of the finite
differences, so this is the function whose gradient the regulariser's jump
terms are).  A spike-time loss adds dl_p/dt_k to the numerator of the jump
at spike k (Table 1 backward transition).

Backward (Table 1 and the Methods): between events the adjoints obey
tau_m lambda_V' = -lambda_V - dl_V/dV and tau_s lambda_I' = -lambda_I + lambda_V
in reverse time; at a spike of neuron n,
  lambda_V <- lambda_V + [theta lambda_V + sum_m w_mn (lambda_V - lambda_I)_m|_{t_k + d_mn}]
                         / (tau_m Vdot^-),   tau_m Vdot^- = I(t_k) - theta;
lambda is continuous at arrivals; and
  dL/dw_ji = -tau_s sum_k lambda_I,j(t_k + d_ji),
  dL/dd_ji = -w_ji  sum_k (lambda_I - lambda_V)_j(t_k + d_ji).
"""
from __future__ import annotations

import heapq
import math
from dataclasses import dataclass, field
from typing import Dict, List, Sequence, Tuple


def _bisect(f, lo, hi, it=200):
    flo = f(lo)
    for _ in range(it):
        mid = 0.5 * (lo + hi)
        fm = f(mid)
        if (fm > 0) == (flo > 0):
            lo, flo = mid, fm
        else:
            hi = mid
        if hi - lo <= 1e-15 * max(1.0, abs(hi)):
            break
    return 0.5 * (lo + hi)


@dataclass
class ContNet:
    """layers: sizes; layer 0 input, 1..L-2 LIF, L-1 LI.  proj: list of
    (pre_layer, post_layer, W[n_pre][n_post], D[n_pre][n_post]) in ms."""
    sizes: Sequence[int]
    proj: List[Tuple[int, int, List[List[float]], List[List[float]]]]
    tau_m: float = 20.0
    tau_s: float = 5.0
    theta: float = 1.0
    T: float = 60.0
    out_lif: bool = False

    def __post_init__(self):
        self.L = len(self.sizes)

    # ----- closed-form free dynamics -------------------------------------------------
    def _kf(self, s):
        tm, ts = self.tau_m, self.tau_s
        return ts / (ts - tm) * (math.exp(-s / ts) - math.exp(-s / tm))

    def _V(self, V, I, s):
        return V * math.exp(-s / self.tau_m) + I * self._kf(s)

    def _dV(self, V, I, s):
        tm, ts = self.tau_m, self.tau_s
        return (-V / tm * math.exp(-s / tm)
                + I * ts / (ts - tm) * (-math.exp(-s / ts) / ts + math.exp(-s / tm) / tm))

    def _intV(self, V, I, s):
        tm, ts = self.tau_m, self.tau_s
        return (V * tm * (1 - math.exp(-s / tm))
                + I * ts / (ts - tm) * (ts * (1 - math.exp(-s / ts)) - tm * (1 - math.exp(-s / tm))))

    def _max_on(self, V, I, s):
        """(max of V on [0, s], argmax); V has at most one extremum."""
        best, arg = V, 0.0
        ve = self._V(V, I, s)
        if ve > best:
            best, arg = ve, s
        d0, d1 = self._dV(V, I, 0.0), self._dV(V, I, s)
        if d0 > 0 > d1:
            r = _bisect(lambda x: self._dV(V, I, x), 0.0, s)
            vr = self._V(V, I, r)
            if vr > best:
                best, arg = vr, r
        return best, arg

    def _crossing(self, V, I, s):
        """First time in (0, s] at which V reaches theta from below, or None."""
        if V >= self.theta:
            return None
        mx, arg = self._max_on(V, I, s)
        if mx < self.theta:
            return None
        return _bisect(lambda x: self._V(V, I, x) - self.theta, 0.0, arg)

    # ----- forward --------------------------------------------------------------------
    def forward(self, in_spikes: Sequence[Tuple[float, int]], loss: str = "integral",
                c: Sequence[float] = None, label: int = 0, delta: float = 0.0,
                lp_lin: Dict[int, float] = None, spike_reg: Dict[int, Tuple[float, float]] = None):
        """in_spikes: (time, input neuron).  Returns (L, record) with record the
        spike list [(t, layer, neuron, I_minus)] and the readout t_max list."""
        assert (loss == "dmse") == self.out_lif
        lp_lin = {} if lp_lin is None else dict(lp_lin)
        spike_reg = {} if spike_reg is None else dict(spike_reg)
        L_ = self.L
        out = L_ - 1
        c = [1.0] * self.sizes[out] if c is None else list(c)
        V = [[0.0] * n for n in self.sizes]
        I = [[0.0] * n for n in self.sizes]
        heap = []
        spikes = []
        seq = [0]

        def emit(t, layer, i):
            for (a, q, W, D) in self.proj:
                if a != layer:
                    continue
                for j in range(self.sizes[q]):
                    ta = t + D[i][j]
                    if ta <= self.T:
                        seq[0] += 1
                        heapq.heappush(heap, (ta, seq[0], q, j, W[i][j]))

        for (t, i) in in_spikes:
            emit(t, 0, i)
        t = 0.0
        integ = [0.0] * self.sizes[out]
        vmax = [0.0] * self.sizes[out]
        tmax = [0.0] * self.sizes[out]
        while True:
            t_next = heap[0][0] if heap else self.T
            t_next = min(t_next, self.T)
            # earliest threshold crossing in (t, t_next]
            tc, who = None, None
            for l in range(1, L_ if self.out_lif else L_ - 1):
                for j in range(self.sizes[l]):
                    x = self._crossing(V[l][j], I[l][j], t_next - t)
                    if x is not None and (tc is None or x < tc):
                        tc, who = x, (l, j)
            step = (tc if tc is not None else t_next - t)
            for k in range(self.sizes[out]):
                integ[k] += self._intV(V[out][k], I[out][k], step)
                mx, arg = self._max_on(V[out][k], I[out][k], step)
                if mx > vmax[k]:
                    vmax[k], tmax[k] = mx, t + arg
            for l in range(1, L_):
                for j in range(self.sizes[l]):
                    V[l][j] = self._V(V[l][j], I[l][j], step)
                    I[l][j] = I[l][j] * math.exp(-step / self.tau_s)
            t = t + step
            if tc is not None:
                l, j = who
                spikes.append((t, l, j, I[l][j]))
                V[l][j] = 0.0
                emit(t, l, j)
                continue
            while heap and heap[0][0] <= t:
                _, _, q, j, w = heapq.heappop(heap)
                I[q][j] += w
            if t >= self.T:
                break
        first = [self.T] * self.sizes[out]
        for (ts_, l, j, _) in spikes:
            if l == out and first[j] == self.T:
                first[j] = ts_
        if loss == "integral":
            Lval = sum(ck * v for ck, v in zip(c, integ))
        elif loss == "max":
            Lval = sum(ck * v for ck, v in zip(c, vmax))
        else:
            Lval = 0.5 * sum((first[i] - first[label] - delta) ** 2
                             for i in range(self.sizes[out]) if i != label)
        Lval += sum(lp_lin.get(l, 0.0) * ts_ for (ts_, l, _, _) in spikes)
        counts = {l: [0] * self.sizes[l] for l in spike_reg}
        for (_, l, j, _) in spikes:
            if l in counts:
                counts[l][j] += 1
        reg_coef = {l: [-rho * (counts[l][j] - nu) for j in range(self.sizes[l])]
                    for l, (rho, nu) in spike_reg.items()}
        Lval += sum(reg_coef[l][j] * ts_ for (ts_, l, j, _) in spikes if l in reg_coef)
        return Lval, {"spikes": spikes, "tmax": tmax, "c": c, "loss": loss, "first": first,
                      "label": label, "delta": delta, "lp_lin": lp_lin, "reg_coef": reg_coef}

    # ----- backward -------------------------------------------------------------------
    def backward(self, in_spikes, rec):
        """Exact EventProp gradients: (dW, dD) lists shaped like proj."""
        L_ = self.L
        out = L_ - 1
        c, loss = rec["c"], rec["loss"]
        tm, ts, th = self.tau_m, self.tau_s, self.theta
        # all spikes (inputs as layer 0)
        allspk = [(t, 0, i, None) for (t, i) in in_spikes] + list(rec["spikes"])
        events = []   # (time, order, kind, payload); processed in descending (time, order)
        for k, (t, l, i, Im) in enumerate(allspk):
            if l > 0:
                events.append((t, 0, "spike", k))
            for p, (a, q, W, D) in enumerate(self.proj):
                if a != l:
                    continue
                for j in range(self.sizes[q]):
                    ta = t + D[i][j]
                    if ta <= self.T:
                        events.append((ta, 1, "arrive", (k, p, i, j)))
        if loss == "max":
            for k in range(self.sizes[out]):
                events.append((rec["tmax"][k], 2, "tmax", k))
        events.sort(key=lambda e: (e[0], e[1]), reverse=True)
        lv = [[0.0] * n for n in self.sizes]
        li = [[0.0] * n for n in self.sizes]
        dW = [[[0.0] * self.sizes[q] for _ in range(self.sizes[a])] for (a, q, _, _) in self.proj]
        dD = [[[0.0] * self.sizes[q] for _ in range(self.sizes[a])] for (a, q, _, _) in self.proj]
        jsum = [0.0] * len(allspk)
        # dl_p / dt_k of every spike: the time-invariant MSE at the first
        # spike of each output neuron, and the linear spike-time terms
        dlp = [0.0] * len(allspk)
        lp_lin = rec.get("lp_lin", {})
        reg_coef = rec.get("reg_coef", {})
        seen = set()
        for k, (tk, l, i, _) in enumerate(allspk):
            if l == 0:
                continue
            dlp[k] += lp_lin.get(l, 0.0)
            if l in reg_coef:
                dlp[k] += reg_coef[l][i]
            if loss == "dmse" and l == out and i not in seen:
                seen.add(i)
                f, lab, dl = rec["first"], rec["label"], rec["delta"]
                if i != lab:
                    dlp[k] += f[i] - f[lab] - dl
                else:
                    dlp[k] -= sum(f[m] - f[lab] - dl for m in range(self.sizes[out]) if m != lab)
        t = self.T

        def propagate(s):
            for l in range(1, L_):
                for j in range(self.sizes[l]):
                    src = c[j] if (l == out and loss == "integral") else 0.0
                    a0 = lv[l][j] + src
                    ev_m, ev_s = math.exp(-s / tm), math.exp(-s / ts)
                    li[l][j] = (li[l][j] * ev_s + a0 * tm / (tm - ts) * (ev_m - ev_s)
                                - src * (1 - ev_s))
                    lv[l][j] = a0 * ev_m - src

        for (te, _, kind, pl) in events:
            propagate(t - te)
            t = te
            if kind == "arrive":
                k, p, i, j = pl
                a, q, W, D = self.proj[p]
                dW[p][i][j] += -ts * li[q][j]
                dD[p][i][j] += -W[i][j] * (li[q][j] - lv[q][j])
                jsum[k] += W[i][j] * (lv[q][j] - li[q][j])
            elif kind == "spike":
                k = pl
                tk, l, i, Im = allspk[k]
                lv[l][i] += (th * lv[l][i] + jsum[k] + dlp[k]) / (Im - th)
            else:
                lv[out][pl] -= c[pl] / tm
        propagate(t)
        return dW, dD

    # ----- finite differences ---------------------------------------------------------
    def fd(self, in_spikes, loss="integral", c=None, h=1e-6, **kw):
        dW = [[[0.0] * self.sizes[q] for _ in range(self.sizes[a])] for (a, q, _, _) in self.proj]
        dD = [[[0.0] * self.sizes[q] for _ in range(self.sizes[a])] for (a, q, _, _) in self.proj]
        for p, (a, q, W, D) in enumerate(self.proj):
            for i in range(self.sizes[a]):
                for j in range(self.sizes[q]):
                    for M, G in ((W, dW), (D, dD)):
                        x0 = M[i][j]
                        M[i][j] = x0 + h
                        lp, _ = self.forward(in_spikes, loss, c, **kw)
                        M[i][j] = x0 - h
                        lm, _ = self.forward(in_spikes, loss, c, **kw)
                        M[i][j] = x0
                        G[p][i][j] = (lp - lm) / (2 * h)
        return dW, dD
