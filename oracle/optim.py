"""Optimiser step of the training loop, as plainly defined (TEST
INFRASTRUCTURE ONLY: the checker, not the product).

The paper trains weights and delays with separate learning rates and
schedules (Methods / "Implementation", hyper-parameter tables) and keeps the
delays non-negative (Fig. 3 caption); it does not name the optimiser.  Two
are defined here, in fp64 on the given arrays:

* SGD:  x <- x - lr g.
* Adam (Kingma & Ba, 2015, Algorithm 1): at step k,
  m <- b1 m + (1 - b1) g,  v <- b2 v + (1 - b2) g^2,
  x <- x - lr (m / (1 - b1^k)) / (sqrt(v / (1 - b2^k)) + eps).

Delays are then clamped to [d_min, d_max] (steps).  The state of every
parameter is independent of every other, so a flat array per tensor is all
that is needed.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional, Sequence

import numpy as np


def sgd(x, g, lr):
    return np.asarray(x, np.float64) - float(lr) * np.asarray(g, np.float64)


@dataclass
class AdamState:
    """First and second moments of one tensor, and the step count."""
    m: np.ndarray
    v: np.ndarray
    k: int = 0


def adam_init(shape) -> AdamState:
    return AdamState(np.zeros(shape, np.float64), np.zeros(shape, np.float64), 0)


def adam(x, g, lr, st: AdamState, b1=0.9, b2=0.999, eps=1e-8):
    """One Adam step of x (returned, fp64); st is advanced in place."""
    g = np.asarray(g, np.float64)
    st.k += 1
    st.m = b1 * st.m + (1.0 - b1) * g
    st.v = b2 * st.v + (1.0 - b2) * g * g
    mhat = st.m / (1.0 - b1 ** st.k)
    vhat = st.v / (1.0 - b2 ** st.k)
    return np.asarray(x, np.float64) - float(lr) * mhat / (np.sqrt(vhat) + eps)


def clamp_delays(D, d_min, d_max):
    return np.clip(np.asarray(D, np.float64), d_min, d_max)


@dataclass
class Optimiser:
    """SGD or Adam over lists of weight and delay tensors (one per
    projection), with per-projection learning-rate factors and the delay
    clamp; fp64 throughout."""
    kind: str                         # "sgd" or "adam"
    b1: float = 0.9
    b2: float = 0.999
    eps: float = 1e-8
    sw: List[AdamState] = field(default_factory=list)
    sd: List[AdamState] = field(default_factory=list)

    def step(self, W: Sequence[np.ndarray], D: Sequence[np.ndarray], dW, dD, lr_w, lr_d,
             d_min, d_max, scale_w: Optional[Sequence[float]] = None,
             scale_d: Optional[Sequence[float]] = None):
        P = len(W)
        scale_w = [1.0] * P if scale_w is None else scale_w
        scale_d = [1.0] * P if scale_d is None else scale_d
        if self.kind == "adam" and not self.sw:
            self.sw = [adam_init(np.shape(w)) for w in W]
            self.sd = [adam_init(np.shape(d)) for d in D]
        outW, outD = [], []
        for p in range(P):
            lw, ld = lr_w * scale_w[p], lr_d * scale_d[p]
            if self.kind == "sgd":
                w, d = sgd(W[p], dW[p], lw), sgd(D[p], dD[p], ld)
            else:
                w = adam(W[p], dW[p], lw, self.sw[p], self.b1, self.b2, self.eps)
                d = adam(D[p], dD[p], ld, self.sd[p], self.b1, self.b2, self.eps)
            outW.append(w)
            outD.append(clamp_delays(d, d_min, d_max))
        return outW, outD
